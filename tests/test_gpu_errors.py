"""Errors found on the device (the error table of the C ABI): a non-finite
input latches CKV_ERR_NONFINITE, returned by ckv_sync or by the next call;
a grid-wide wait that gives up (forced from the host with a zero barrier
bound) makes the joint test report n_accepted = -1, the grid selection
n_kept = -1, and the lifecycle driver return its error -- every kernel
still exits normally."""
import numpy as np
import pytest
import torch

from synth import WORKLOADS, make_layer, scaled
from tests.gpu_util import LayerOnDevice

pytestmark = pytest.mark.gpu

NONFINITE, UNSUPPORTED = -7, -4


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _views(P, dl, k=None, v=None):
    kv = P.kv_view(dl.k if k is None else k, dl.v if v is None else v, dl.pos)
    win = P.window_view(dl.q_post, dl.qpos_post)
    pages = P.Pages(dl.L.layout.page_start, dl.L.layout.page_len)
    return kv, win, pages


@pytest.mark.parametrize("which", ["key", "value", "recorded", "recorded_lse_no_pages"])
def test_nonfinite_input_is_latched(ckv, which):
    P, ctx = ckv
    L = make_layer(WORKLOADS["tiny"], seed=2)
    dl = LayerOnDevice(L)
    print(f"[errors] non-finite {which}", flush=True)
    kv, win, pages = _views(P, dl)
    ctx.sync()                                   # nothing latched before
    if which == "recorded":
        m = P.ckv_measure_page_effects(ctx, kv, win, pages, want=("R", "o", "lse"))
        o = m["o"].reshape(-1).clone()
        o[5] = float("nan")
        P.ckv_measure_recorded(ctx, kv, win, pages, o, m["lse"].reshape(-1).contiguous())
    elif which == "recorded_lse_no_pages":
        # a recorded log-sum-exp of -inf for a row that sees tokens, in a call
        # without pages (token mass only): the mass of its tokens is infinite
        m = P.ckv_measure_page_effects(ctx, kv, win, pages, want=("R", "o", "lse"))
        lse = m["lse"].reshape(-1).clone()
        lse[3] = float("-inf")
        P.ckv_measure_recorded(ctx, kv, win, P.Pages(np.zeros(0, np.int32), np.zeros(0, np.int32)),
                               m["o"].reshape(-1).contiguous(), lse, want=("token_mass",))
    else:
        k, v = dl.k.clone(), dl.v.clone()
        t = int(L.layout.page_start[3])          # a token every post-window row sees
        (k if which == "key" else v)[0, t, 7] = float("nan")
        kv2, _, _ = _views(P, dl, k, v)
        P.ckv_measure_page_effects(ctx, kv2, win, pages)
    with pytest.raises(P.CKVError) as e:
        ctx.sync()
    assert e.value.code == NONFINITE
    ctx.sync()                                   # reported once, then cleared
    P.ckv_measure_page_effects(ctx, kv, win, pages)
    ctx.sync()


def test_nonfinite_reported_by_next_call(ckv):
    P, ctx = ckv
    L = make_layer(WORKLOADS["tiny"], seed=3)
    dl = LayerOnDevice(L)
    kv, win, pages = _views(P, dl)
    k = dl.k.clone()
    k[0, int(L.layout.page_start[0]), 0] = float("inf")
    kv2, _, _ = _views(P, dl, k)
    P.ckv_measure_page_effects(ctx, kv2, win, pages)
    torch.cuda.synchronize()                     # the kernels have finished
    with pytest.raises(P.CKVError) as e:
        P.ckv_measure_page_effects(ctx, kv, win, pages)
    assert e.value.code == NONFINITE
    P.ckv_measure_page_effects(ctx, kv, win, pages)
    ctx.sync()


def test_barrier_give_up_joint_and_selection(ckv):
    """A zero barrier bound: the first workgroup to reach a grid-wide wait
    gives up, every workgroup leaves, the counts read -1; with the default
    bound restored, the same calls succeed (the persistent selection state
    was left clean)."""
    P, ctx = ckv
    w = scaled("stress", n_tokens=4096, n_q_heads=8, n_kv_heads=2, max_cand=64)
    L = make_layer(w, seed=5)
    dl = LayerOnDevice(L)
    kv, win, pages = _views(P, dl)
    m = P.ckv_measure_page_effects(ctx, kv, win, pages, want=("R", "o", "lse"))
    cl = P.ckv_classify_pages(ctx, m["R"], m["R"], force=torch.tensor(L.forced.astype(np.uint8)).cuda(),
                              max_cand=64)
    S = w.n_tokens
    k5, v5 = dl.k[None, None], dl.v[None, None]
    score = torch.rand((1, S), device="cuda")

    def run():
        jt = P.ckv_joint_test(ctx, kv, win, m["o"].reshape(-1), m["lse"].reshape(-1), pages, cl["cand"],
                              cl["n_cand"], 64, 0.01)
        sel = P.ckv_select_and_compact(ctx, k5, v5, dl.pos[None], [S], score, [P.Pages([], [])],
                                       [P.Pages([], [])], [None], budget=1024)
        torch.cuda.synchronize()
        return int(jt["n_accepted"].item()), int(sel["n_kept"][0].item())

    ctx.set_barrier_timeout_us(0)
    try:
        na, nk = run()
    finally:
        ctx.set_barrier_timeout_us(1342177)
    print(f"[errors] zero bound: n_accepted {na} n_kept {nk}", flush=True)
    assert na == -1 and nk == -1
    na, nk = run()
    assert na >= 0 and nk == 1024


def test_barrier_give_up_agent(ckv):
    """The lifecycle driver turns a joint test that gave up into an error:
    with a zero barrier bound around every post-commit step of tiny agent
    episodes (the trajectory's own keys, values and queries, with forced
    high-to-low pages), the first step that has candidates to test fails
    with CKV_ERR_UNSUPPORTED."""
    P, ctx = ckv
    from synth.trajectory import TRAJECTORIES, kv_rows, make_trajectory, query_rows, schedule
    from tests.gpu_util import dev_bf16, dev_i32
    cfg = TRAJECTORIES["tiny_agent"]
    failed = None
    for seed in (3, 4, 5, 6):
        traj = make_trajectory(cfg, seed=seed, n_turns=8)
        ag = P.Agent(ctx, cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, cfg.capacity, page_size=cfg.page_size,
                     window=cfg.window, n_q_heads=cfg.n_q_heads, budget=cfg.budget, eta=cfg.eta,
                     max_pending_pages=cfg.max_pending_pages, keep_recent=cfg.keep_recent,
                     max_scan_pages=cfg.max_scan_pages, checkpoint_every=cfg.checkpoint_every,
                     score_layer=cfg.score_layer)
        try:
            for act in schedule(traj):
                if act[0] == "append":
                    _, kind, p0, p1, dec, first = act
                    kv = [kv_rows(traj, l, p0, p1) for l in range(cfg.n_layers)]
                    ag.append(kind, dev_bf16(np.stack([x[0] for x in kv])), dev_bf16(np.stack([x[1] for x in kv])),
                              np.arange(p0, p1), dec, first)
                    continue
                p0 = act[1]
                q = dev_bf16(query_rows(traj, cfg.score_layer, p0, p0 + cfg.window))
                qp = dev_i32(np.arange(p0, p0 + cfg.window))
                if act[0] != "post":
                    getattr(ag, act[0])(q, qp)
                    continue
                ctx.set_barrier_timeout_us(0)
                try:
                    ag.post(q, qp)
                except P.CKVError as e:
                    failed = e
                finally:
                    ctx.set_barrier_timeout_us(1342177)
                if failed is not None:
                    break
        finally:
            ag.close()
        if failed is not None:
            break
    print(f"[errors] agent: {failed}", flush=True)
    assert failed is not None and failed.code == UNSUPPORTED, failed
