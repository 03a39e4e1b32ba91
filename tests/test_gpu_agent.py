"""GPU parity of the lifecycle driver (include/commitkv_agent.h, Algorithm 1)
against the oracle driver (oracle/lifecycle.py), step by step over whole
synthetic agent episodes.

The library's agent and the oracle's run the same schedule in lock step.  At
every step the GPU's outputs are checked against the oracle's computation
from the same state, then the oracle adopts the GPU's values where the
single-call parity bars allow them to differ, so that both keep one state:
  commit      identical page lists (E_c, scan cap); R^- within 2e-3; the
              oracle then keeps the GPU's float32 R^-;
  post        identical measured pages; R^+ within 2e-3; states and candidate
              order identical to the oracle's classification of the GPU's
              float32 effects; union effects replayed along the GPU's
              decisions within 2e-3 and every decision equal to the replayed
              gate unless within 2e-3 of tau; D_c identical;
  checkpoint  the same decision to compact; base score (token mass) within
              3e-3; kept indices identical to the oracle's selection on the
              GPU's float32 scores; every layer's compacted keys, values and
              positions bit-exact against the oracle's cache.
Due flags reported by ckv_agent_append must match the schedule.
"""
import numpy as np
import pytest
import torch

import oracle as O
from synth.trajectory import (TRAJECTORIES, kv_rows, make_trajectory, query_rows, schedule,
                              scaled_trajectory)
from tests.agent_util import oracle_agent
from tests.gpu_util import REL_TOL, assert_scores_close, dev_bf16, dev_i32

pytestmark = pytest.mark.gpu

TH32 = {k: float(np.float32(v)) for k, v in O.PAPER_THRESHOLDS.items()}


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.set_policy()
    ctx.close()


def _gpu_agent(P, ctx, cfg, paged=None, spare_rows=37):
    """paged: None for the two-buffer agent, else the row seed of a paged
    agent whose pool has spare_rows more rows than the capacity."""
    extra = {} if paged is None else dict(paged=True, pool_rows=cfg.capacity + spare_rows, row_seed=paged)
    return P.Agent(ctx, cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, cfg.capacity,
                   page_size=cfg.page_size, window=cfg.window, n_q_heads=cfg.n_q_heads,
                   budget=cfg.budget, eta=cfg.eta, max_pending_pages=cfg.max_pending_pages,
                   keep_recent=cfg.keep_recent, max_scan_pages=cfg.max_scan_pages,
                   checkpoint_every=cfg.checkpoint_every, score_layer=cfg.score_layer,
                   report_detail=True, pool_kernel=cfg.pool_kernel, pool_mode=cfg.pool_mode, **extra)


def _expected_due(acts, i):
    """Flags the append at acts[i] must report: the actions up to the next append."""
    due = 0
    for a in acts[i + 1:]:
        if a[0] == "append":
            break
        due |= {"post": 1, "checkpoint": 2}.get(a[0], 0)
    return due


def _check_cache(ga, oa, cfg):
    k, v, pos, n = ga.cache()
    assert n == oa.pos.size
    if ga.paged:
        rows = ga.rows("resident")
        assert rows.size == n and np.unique(rows).size == n
        assert sorted(ga.free + rows.tolist()) == list(range(ga.kp.shape[2]))
    np.testing.assert_array_equal(pos[:n].cpu().numpy(), oa.pos)
    kb = k[:, :, :n].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    vb = v[:, :, :n].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    for l in range(cfg.n_layers):
        np.testing.assert_array_equal(kb[l], oa.K[l])
        np.testing.assert_array_equal(vb[l], oa.V[l])


def run_lockstep(P, ctx, traj, ablation=(), paged=None, spare_rows=37):
    cfg = traj.cfg
    ga = _gpu_agent(P, ctx, cfg, paged, spare_rows)
    oa = oracle_agent(cfg, ablation=ablation)
    acts = schedule(traj)
    stats = dict(commit=0, post=0, cand=0, accepted=0, compacted=0, excused=0)
    try:
        for i, act in enumerate(acts):
            if act[0] == "append":
                _, kind, p0, p1, dec, first = act
                kv = [kv_rows(traj, l, p0, p1) for l in range(cfg.n_layers)]
                kd = dev_bf16(np.stack([x[0] for x in kv]))
                vd = dev_bf16(np.stack([x[1] for x in kv]))
                due = ga.append(kind, kd, vd, np.arange(p0, p1), dec, first)
                oa.append(kind, p0, p1, [x[0] for x in kv], [x[1] for x in kv], dec, first)
                assert due == _expected_due(acts, i), (i, act, due)
                continue
            p0 = act[1]
            Qb = query_rows(traj, cfg.score_layer, p0, p0 + cfg.window)
            qpos = np.arange(p0, p0 + cfg.window)
            q, qp = dev_bf16(Qb), dev_i32(qpos)
            print(f"[agent] step {i} {act[0]} at {p0}: resident {oa.pos.size}", flush=True)
            if act[0] == "commit":
                g = ga.commit(q, qp)
                o = oa.commit(Qb, qpos)
                assert g["pages"] == o["pages"]
                assert_scores_close(g["R_pre"], o["R_pre"], "R_pre")
                oa.pending = (o["pages"], g["R_pre"].astype(np.float64))
                stats["commit"] += 1
            elif act[0] == "post":
                g = ga.post(q, qp)
                m = oa.post_measure(Qb, qpos)
                assert g["pages"] == m["pages"]
                np.testing.assert_array_equal(g["R_pre"], m["R_pre"].astype(np.float32))
                if m["pages"]:
                    assert_scores_close(g["R_post"], m["R_post"], "R_post")
                    th = {k: TH32[k] for k in ("tau_use", "tau_dead", "rho_use", "rho_dead")}
                    lam, _, _, cand = O.classify(g["R_pre"].astype(np.float64), g["R_post"].astype(np.float64),
                                                 [s for s, _ in oa.ranges(m["pages"])], ablation=ablation, **th)
                    np.testing.assert_array_equal(g["lam"], lam)
                    np.testing.assert_array_equal(g["cand"], cand)
                if len(g["cand"]):
                    K, V, pos = oa._layer()
                    ref = O.joint_replay(K, V, pos, Qb, qpos, oa.ranges(m["pages"]), g["cand"].tolist(),
                                         g["accepted"].astype(bool).tolist(), method="closed")
                    assert_scores_close(g["union_R"], ref, "union_R")
                    tau = TH32["tau_joint"]
                    for a, r in zip(g["accepted"], ref):
                        if abs(r - tau) <= REL_TOL * tau:
                            stats["excused"] += 1
                            continue
                        if "no_joint" in ablation:
                            assert a == 1
                        else:
                            assert bool(a) == (r <= tau), (a, r)
                acc = [m["pages"][c] for c, a in zip(g["cand"], g["accepted"]) if a]
                oa.retire(acc)
                oa.end_commit()
                assert [tuple(p) for p in ga.pages("retired")] == oa.retired
                stats["post"] += 1
                stats["cand"] += len(g["cand"])
                stats["accepted"] += int(g["n_accepted"])
            else:
                g = ga.checkpoint(q, qp)
                S = oa.pos.size
                _, _, ret = oa.checkpoint_lists()
                assert g["compacted"] == (S > cfg.budget or bool(ret))
                if g["compacted"]:
                    want = oa.base_score(Qb, qpos)
                    np.testing.assert_allclose(g["score"], want, rtol=3e-3, atol=1e-6)
                    c = oa.checkpoint(Qb, qpos, score=g["score"])
                    np.testing.assert_array_equal(g["kept"], c["kept"])
                    _check_cache(ga, oa, cfg)
                    stats["compacted"] += 1
        n, _, dec = ga.state()
        assert n == oa.pos.size and dec == oa.decoded
    finally:
        ga.close()
    print(f"[agent] {traj.cfg.name} seed {traj.seed}: {stats}", flush=True)
    return stats


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tiny_episode(ckv, seed):
    P, ctx = ckv
    traj = make_trajectory(TRAJECTORIES["tiny_agent"], seed=seed, n_turns=8)
    s = run_lockstep(P, ctx, traj)
    assert s["compacted"] >= 2 and s["post"] >= 5


def test_tiny_episodes_cover_retirement(ckv):
    """Across a few seeds the forced pages become candidates and are retired
    by the driver (the joint test and D_c are exercised, not only empty lists)."""
    P, ctx = ckv
    tot = dict(cand=0, accepted=0)
    for seed in (3, 4):
        s = run_lockstep(P, ctx, make_trajectory(TRAJECTORIES["tiny_agent"], seed=seed, n_turns=8))
        tot["cand"] += s["cand"]
        tot["accepted"] += s["accepted"]
    assert tot["cand"] >= 3 and tot["accepted"] >= 2


def test_paper_operating_point_episode(ckv):
    """The paper's settings (W=8, G=16, eta=0.125, <= 64 scanned pages, <= 16
    protected, checkpoints every 128 decoded tokens) on a Qwen3-14B-shaped
    layer (40 query / 8 KV heads, d=128; 5 query heads per KV head), budget
    2048, two layers, a short episode with forced transitions."""
    P, ctx = ckv
    cfg = scaled_trajectory("paper_agent", n_layers=2, score_layer=1, budget=2048, obs_hi=768,
                            reason_hi=384, prompt_hi=512, forced_frac=0.1, forced_pre=100.0,
                            forced_post=0.005, heavy_frac=0.003)
    s = run_lockstep(P, ctx, make_trajectory(cfg, seed=0, n_turns=6))
    assert s["compacted"] >= 1 and s["commit"] >= 5


@pytest.mark.parametrize("budget,turns,obs_hi", [(4096, 9, 1024), (8192, 12, 1536)])
def test_paper_operating_point_budgets(ckv, budget, turns, obs_hi):
    """The paper's other two budgets (Sec. 4.1) at its operating point, each
    episode long enough that checkpoints compact the cache past the budget."""
    P, ctx = ckv
    cfg = scaled_trajectory("paper_agent", n_layers=2, score_layer=1, budget=budget, obs_hi=obs_hi,
                            reason_hi=384, prompt_hi=512, forced_frac=0.1, forced_pre=100.0,
                            forced_post=0.005, heavy_frac=0.003)
    traj = make_trajectory(cfg, seed=0, n_turns=turns)
    assert traj.n_tokens > budget + 256
    s = run_lockstep(P, ctx, traj)
    assert s["compacted"] >= 1 and s["commit"] >= turns - 1


@pytest.mark.parametrize("mode", ["max", "mean"])
def test_pooled_score_episode(ckv, mode):
    """The SnapKV-style pooled base score (7 tokens) at every checkpoint."""
    P, ctx = ckv
    cfg = scaled_trajectory("tiny_agent", pool_kernel=7, pool_mode=mode)
    s = run_lockstep(P, ctx, make_trajectory(cfg, seed=5, n_turns=6))
    assert s["compacted"] >= 2


@pytest.mark.parametrize("seed", [0, 3])
def test_paged_episode(ckv, seed):
    """A paged agent (slot table over scattered pool rows, checkpoints that
    move no key or value) in lock step with the oracle: the same bars as the
    two-buffer agent; the resident rows, gathered, must equal the oracle's
    cache bit for bit, and every pool row is either resident or free."""
    P, ctx = ckv
    s = run_lockstep(P, ctx, make_trajectory(TRAJECTORIES["tiny_agent"], seed=seed, n_turns=8), paged=seed + 11)
    assert s["compacted"] >= 2 and s["post"] >= 5


def test_paged_tight_pool_episode(ckv):
    """A pool of exactly the capacity: after the first checkpoints every
    append reuses rows that a checkpoint freed, in scattered order."""
    P, ctx = ckv
    s = run_lockstep(P, ctx, make_trajectory(TRAJECTORIES["tiny_agent"], seed=4, n_turns=8), paged=9,
                     spare_rows=0)
    assert s["compacted"] >= 2


def test_paged_paper_operating_point_episode(ckv):
    """The paper's operating point (W 8, G 16, a Qwen3-14B-shaped layer)
    through a paged agent."""
    P, ctx = ckv
    cfg = scaled_trajectory("paper_agent", n_layers=2, score_layer=1, budget=2048, obs_hi=768,
                            reason_hi=384, prompt_hi=512, forced_frac=0.1, forced_pre=100.0,
                            forced_post=0.005, heavy_frac=0.003)
    s = run_lockstep(P, ctx, make_trajectory(cfg, seed=1, n_turns=6), paged=5)
    assert s["compacted"] >= 1 and s["commit"] >= 5


def test_paged_ablation_episode(ckv):
    P, ctx = ckv
    ctx.set_policy("no_protection")
    try:
        run_lockstep(P, ctx, make_trajectory(TRAJECTORIES["tiny_agent"], seed=2, n_turns=6), ("no_protection",),
                     paged=3)
    finally:
        ctx.set_policy()


def test_paged_pooled_episode(ckv):
    P, ctx = ckv
    cfg = scaled_trajectory("tiny_agent", pool_kernel=7, pool_mode="max")
    s = run_lockstep(P, ctx, make_trajectory(cfg, seed=5, n_turns=6), paged=2)
    assert s["compacted"] >= 2


@pytest.mark.parametrize("ablation", [("no_protection",), ("no_joint",), ("no_precommit",)])
def test_ablation_episode(ckv, ablation):
    P, ctx = ckv
    ctx.set_policy(*ablation)
    try:
        run_lockstep(P, ctx, make_trajectory(TRAJECTORIES["tiny_agent"], seed=1, n_turns=6), ablation)
    finally:
        ctx.set_policy()


def test_host_errors(ckv):
    P, ctx = ckv
    cfg = TRAJECTORIES["tiny_agent"]
    ga = _gpu_agent(P, ctx, cfg)
    try:
        k = torch.zeros((cfg.n_layers, cfg.n_kv_heads, 4, cfg.head_dim), dtype=torch.bfloat16, device="cuda")
        ga.append(3, k, k, np.arange(10, 14), False)
        with pytest.raises(P.CKVError) as e:          # positions must increase
            ga.append(3, k, k, np.arange(0, 4), False)
        assert e.value.code == -1
        with pytest.raises(P.CKVError) as e:          # inside an event positions are consecutive
            ga.append(3, k, k, np.array([20, 21, 23, 24]), False, begins_event=False)
        assert e.value.code == -1
        q = torch.zeros((cfg.n_q_heads, cfg.window + 1, cfg.head_dim), dtype=torch.bfloat16, device="cuda")
        with pytest.raises(P.CKVError) as e:          # window rows differ from the configuration
            ga.commit(q, dev_i32(np.arange(cfg.window + 1)))
        assert e.value.code == -2
        r = ga.post(q[:, :cfg.window], dev_i32(np.arange(cfg.window)))   # no pending commit: nothing
        assert r["op"] == 2 and r["pages"] == []
    finally:
        ga.close()
    with pytest.raises(P.CKVError) as e:
        P.Agent(ctx, 2, 1, 64, 256, page_size=16, window=16, n_q_heads=4, budget=512)   # B > capacity
    assert e.value.code == -1


def test_paged_host_errors(ckv):
    import ctypes
    from paper_2608_07855_amd import _abi
    P, ctx = ckv
    cfg = TRAJECTORIES["tiny_agent"]
    ga = _gpu_agent(P, ctx, cfg, paged=0)
    gb = _gpu_agent(P, ctx, cfg)
    L = P.lib()
    try:
        pos = np.arange(4, dtype=np.int32)
        bad = np.array([0, 1, ga.kp.shape[2], 3], np.int32)          # a row outside the pool
        i32 = lambda a: a.ctypes.data_as(_abi.c_i32p)
        assert L.ckv_agent_append_rows(ga.handle, 3, i32(pos), i32(bad), 4, 0, 1, None) == _abi.CKV_ERR_ARG
        assert L.ckv_agent_append(ga.handle, 3, i32(pos), 4, 0, 1, None) == _abi.CKV_ERR_ARG
        assert L.ckv_agent_append_rows(gb.handle, 3, i32(pos), i32(pos), 4, 0, 1, None) == _abi.CKV_ERR_ARG
        n = ctypes.c_int32()
        assert L.ckv_agent_rows(gb.handle, 0, None, 0, ctypes.byref(n)) == _abi.CKV_ERR_ARG
        assert ga.state()[0] == 0 and ga.rows("resident").size == 0
        k = torch.zeros((cfg.n_layers, cfg.n_kv_heads, 4, cfg.head_dim), dtype=torch.bfloat16, device="cuda")
        ga.append(3, k, k, pos, False)
        assert ga.rows("pos").tolist() == pos.tolist() and ga.rows("resident").size == 4
    finally:
        ga.close()
        gb.close()
    with pytest.raises(P.CKVError) as e:                           # capacity above the pool's rows
        P.Agent(ctx, 2, 1, 64, 512, page_size=16, window=16, n_q_heads=4, budget=256, paged=True, pool_rows=300)
    assert e.value.code == -2
