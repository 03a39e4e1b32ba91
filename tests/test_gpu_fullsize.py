"""Full-size parity, in the launch configuration the benchmark times.

* the Qwen3-8B-shaped layer and the joint-test stress layer (32768 tokens):
  R and R_head of every page on every query head, pre and post, against the
  oracle's closed form stored in ``tests/golden/fullsize_<workload>.npz``
  (written by ``tests/golden/make_fullsize.py`` from ``oracle/`` only; the
  inputs' digest is checked first); the lifecycle states from the GPU's own
  effects against the oracle's states, except for pages whose effect or
  percentile sits within the tolerance of a threshold; window outputs of
  sampled heads; the token window-mass of every token;
* the Qwen3-32B-shaped layer (131072 tokens, 128-row windows, 64-token
  pages): per-head effects of every page for one query head;
* the joint-test stress layer (30% forced pages, 256 candidates): every
  union effect of the greedy sequence replayed by the oracle's closed form
  of Eq. (6) over the union, and every decision checked;
* the 36-layer x 4-sequence stack at 65536 tokens: kept indices bit-exact
  against the oracle's selection, compacted bytes checked on sampled
  (sequence, layer, head) slices.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
from synth import WORKLOADS, make_layer, make_scores
from tests.gpu_util import REL_TOL, LayerOnDevice, assert_scores_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _measure(P, ctx, dl, which, want):
    L = dl.L
    if which == "pre":
        kv = P.kv_view(dl.k, dl.v, dl.pos, n_tokens=L.layout.s_pre)
        win = P.window_view(dl.q_pre, dl.qpos_pre)
    else:
        kv = P.kv_view(dl.k, dl.v, dl.pos)
        win = P.window_view(dl.q_post, dl.qpos_post)
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    out = P.ckv_measure_page_effects(ctx, kv, win, pages, want=want)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if torch.is_tensor(v) else v) for k, v in out.items()}


def _oracle_heads(L, which, heads):
    S = L.layout.s_pre if which == "pre" else L.w.n_tokens
    q = L.q_pre if which == "pre" else L.q_post
    qpos = L.qpos_pre if which == "pre" else L.qpos_post
    _, Rh = O.page_effects(L.k[:, :S], L.v[:, :S], L.pos[:S], q, qpos, L.pages,
                           method="closed", heads=heads)
    return Rh


@pytest.fixture(scope="module")
def q8b():
    L = make_layer(WORKLOADS["q8b"], seed=0)
    return L, LayerOnDevice(L)


def _golden(L, name):
    import os
    from tests.golden.make_fullsize import input_digest
    path = os.path.join(os.path.dirname(__file__), "golden", f"fullsize_{name}.npz")
    g = np.load(path, allow_pickle=False)
    assert str(g["digest"]) == input_digest(L), f"{path}: the synthetic inputs changed; regenerate it"
    return g


@pytest.fixture(scope="module")
def stress():
    L = make_layer(WORKLOADS["stress"], seed=0)
    return L, LayerOnDevice(L)


@pytest.mark.parametrize("which", ["pre", "post"])
@pytest.mark.parametrize("name", ["q8b", "stress"])
def test_fullsize_every_head_golden(ckv, q8b, stress, name, which):
    """R and R_head of every page on all 32 query heads at 32768 tokens."""
    P, ctx = ckv
    L, dl = q8b if name == "q8b" else stress
    g = _golden(L, name)
    print(f"[fullsize] {name} {which}: S={L.w.n_tokens} pages={len(L.pages)} all {L.w.n_q_heads} heads",
          flush=True)
    got = _measure(P, ctx, dl, which, ("R", "R_head"))
    assert_scores_close(got["R_head"], g[f"R_head_{which}"], f"{name} {which} R_head (every head)")
    assert_scores_close(got["R"], g[f"R_{which}"], f"{name} {which} R")


@pytest.mark.parametrize("name", ["q8b", "stress"])
def test_fullsize_states(ckv, q8b, stress, name):
    """Lifecycle states at 32768 tokens (Eq. (8)-(10)) from the GPU's own
    effects, against the oracle's states from its effects: identical except
    for pages whose effect lies within the tolerance of a tau or whose
    percentile band contains a rho."""
    from tests.test_gpu_classify import TH, _excused
    P, ctx = ckv
    L, dl = q8b if name == "q8b" else stress
    g = _golden(L, name)
    pre = _measure(P, ctx, dl, "pre", ("R",))["R"]
    post = _measure(P, ctx, dl, "post", ("R",))["R"]
    out = P.ckv_classify_pages(ctx, torch.from_numpy(pre).cuda(), torch.from_numpy(post).cuda(), TH)
    torch.cuda.synchronize()
    lam = out["lam"].cpu().numpy()
    lam_o, *_ = O.classify(g["R_pre"], g["R_post"], L.layout.page_start, **TH)
    ex = _excused(g["R_pre"], g["R_post"])
    diff = np.flatnonzero((lam != lam_o) & ~ex)
    print(f"[fullsize] {name} states: gpu {np.bincount(lam, minlength=5).tolist()} oracle "
          f"{np.bincount(lam_o, minlength=5).tolist()}; excused {int(ex.sum())}, differing "
          f"{int((lam != lam_o).sum())}", flush=True)
    assert diff.size == 0, f"states differ at {diff[:10]}: gpu {lam[diff[:10]]} oracle {lam_o[diff[:10]]}"


def test_q8b_window_outputs_sampled_heads(ckv, q8b):
    P, ctx = ckv
    L, dl = q8b
    heads = [0, 13, 31]
    for which in ("pre", "post"):
        got = _measure(P, ctx, dl, which, ("R", "o", "lse"))
        S = L.layout.s_pre if which == "pre" else L.w.n_tokens
        q = L.q_pre if which == "pre" else L.q_post
        qpos = L.qpos_pre if which == "pre" else L.qpos_post
        K, V, Q = O.as_f64(L.k[:, :S]), O.as_f64(L.v[:, :S]), O.as_f64(q)
        vis = O.visibility(L.pos[:S], qpos)
        group = L.w.n_q_heads // L.w.n_kv_heads
        for h in heads:
            s = O.head_logits(Q[h], K[h // group], 1.0 / math.sqrt(L.w.head_dim))
            _, o = O.attend(s, vis, V[h // group])
            np.testing.assert_allclose(got["o"][h], o, rtol=0, atol=2e-3 * np.abs(o).max())


def test_q8b_token_mass(ckv, q8b):
    P, ctx = ckv
    L, dl = q8b
    got = _measure(P, ctx, dl, "post", ("R", "token_mass"))
    want = O.token_mass(L.k, L.v, L.pos, L.q_post, L.qpos_post)
    np.testing.assert_allclose(got["token_mass"], want, rtol=3e-3, atol=1e-6)


def test_q32b_sampled_head(ckv):
    P, ctx = ckv
    L = make_layer(WORKLOADS["q32b"], seed=0)
    dl = LayerOnDevice(L)
    print(f"[fullsize] q32b: S={L.w.n_tokens} pages={len(L.pages)}", flush=True)
    for which in ("pre", "post"):
        got = _measure(P, ctx, dl, which, ("R", "R_head"))
        Rh = _oracle_heads(L, which, [40])
        assert_scores_close(got["R_head"][:, 40], Rh[:, 40], f"q32b {which} R_head[:, 40]")


def test_stress_joint_full_replay(ckv, stress):
    """Forced high-to-low pages fed as candidates (capped at 256); every
    union effect R+(A_t u {E_t}) of the greedy sequence is replayed with the
    GPU's own order and decisions.  The oracle's attention (a, o) is computed
    once per query head; each union then goes through the oracle's closed
    form of Eq. (6), evaluated on the candidate pages' tokens plus a block of
    tokens every row sees and no candidate holds (the form reads a only on
    deleted tokens, and the extra block keeps its "a row sees nothing else"
    test exact)."""
    import time
    P, ctx = ckv
    L, dl = stress
    w = L.w
    kv = P.kv_view(dl.k, dl.v, dl.pos)
    win = P.window_view(dl.q_post, dl.qpos_post)
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    kv_pre = P.kv_view(dl.k, dl.v, dl.pos, n_tokens=L.layout.s_pre)
    win_pre = P.window_view(dl.q_pre, dl.qpos_pre)
    pre = P.ckv_measure_page_effects(ctx, kv_pre, win_pre, pages)
    post = P.ckv_measure_page_effects(ctx, kv, win, pages, want=("R", "o", "lse"))
    force = torch.from_numpy(L.forced.astype(np.uint8)).cuda()
    cl = P.ckv_classify_pages(ctx, pre["R"], post["R"], force=force, max_cand=w.max_cand)
    jt = P.ckv_joint_test(ctx, kv, win, post["o"].reshape(-1), post["lse"].reshape(-1), pages,
                          cl["cand"], cl["n_cand"], w.max_cand, 0.01)
    torch.cuda.synchronize()
    n_cand = int(cl["n_cand"].item())
    cand = cl["cand"].cpu().numpy()[:n_cand]
    acc = jt["accepted"].cpu().numpy()[:n_cand]
    uR = jt["union_R"].cpu().numpy()[:n_cand]
    R_post = post["R"].cpu().numpy()
    print(f"[fullsize] stress: candidates {n_cand} accepted {int(acc.sum())}", flush=True)
    lam = cl["lam"].cpu().numpy()
    assert n_cand == min(w.max_cand, int(((lam == O.CANDIDATE) | L.forced).sum()))
    assert_scores_close(uR[:1], R_post[cand[:1]], "union_R[0] vs R+")
    # token columns: every candidate page's tokens, then a block no candidate holds
    S = w.n_tokens
    in_cand = np.zeros(S, bool)
    for j in cand:
        st, ln = L.pages[j]
        in_cand[st:st + ln] = True
    vis = O.visibility(L.pos, L.qpos_post)
    always = np.flatnonzero(~in_cand & vis.all(axis=0))[:64]
    assert always.size > 0
    cols = np.concatenate([np.flatnonzero(in_cand), always])
    page_cols = {}
    for j in cand:
        st, ln = L.pages[j]
        page_cols[int(j)] = np.flatnonzero((cols >= st) & (cols < st + ln))
    K, V, Q = O.as_f64(L.k), O.as_f64(L.v), O.as_f64(L.q_post)
    group = w.n_q_heads // w.n_kv_heads
    ref = np.zeros(n_cand)
    t0 = time.time()
    for h in range(w.n_q_heads):
        g = h // group
        a, o = O.attend(O.head_logits(Q[h], K[g], 1.0 / math.sqrt(w.head_dim)), vis, V[g])
        a_c, v_c, vis_c = a[:, cols], V[g][cols], vis[:, cols]
        delete = np.zeros(cols.size, bool)
        for t, j in enumerate(cand):
            trial = delete.copy()
            trial[page_cols[int(j)]] = True
            r = O.deletion_ratio_closed_form(a_c, o, v_c, trial, vis_c)
            ref[t] = max(ref[t], float(r.max()))
            if acc[t]:
                delete = trial
    print(f"[fullsize] stress replay of {n_cand} steps over {w.n_q_heads} heads in {time.time() - t0:.1f}s",
          flush=True)
    assert_scores_close(uR, ref, "union_R (every step)")
    for t in range(n_cand):
        if abs(ref[t] - 0.01) > REL_TOL * 0.01:
            assert bool(acc[t]) == (ref[t] <= 0.01), f"step {t}: R_ref={ref[t]}"


def test_stack_compaction_sampled(ckv):
    """36 layers x 4 sequences at 65536 tokens, budget 16384: kept indices
    bit-exact, compacted K/V/positions checked on sampled slices."""
    P, ctx = ckv
    w = WORKLOADS["q8b_stack"]
    ns, nl, H, S, d, B = w.n_seq, w.n_layers, w.n_kv_heads, w.n_tokens, w.head_dim, w.budget
    g = torch.Generator(device="cuda").manual_seed(7)
    k = torch.randint(-32768, 32767, (ns, nl, H, S, d), dtype=torch.int16, device="cuda", generator=g)
    v = torch.randint(-32768, 32767, (ns, nl, H, S, d), dtype=torch.int16, device="cuda", generator=g)
    pos_np = np.stack([np.arange(S, dtype=np.int32) * (s + 1) for s in range(ns)])
    pos = torch.from_numpy(pos_np).cuda()
    score = np.stack([make_scores(S, seed=40 + s) for s in range(ns)])
    rng = np.random.default_rng(3)
    retired, pending, rpre = [], [], []
    for s in range(ns):
        st = np.sort(rng.choice(S // 64, 48, replace=False)) * 64
        ln = rng.integers(1, 65, 48)
        pages = list(zip(st.tolist(), ln.tolist()))
        retired.append(pages[:24])
        pending.append(pages[24:])
        rpre.append(rng.uniform(0, 1, 24).astype(np.float32))
    out = P.ckv_select_and_compact(
        ctx, k.view(torch.bfloat16), v.view(torch.bfloat16), pos, [S] * ns, torch.from_numpy(score).cuda(),
        [P.Pages([p[0] for p in r], [p[1] for p in r]) for r in retired],
        [P.Pages([p[0] for p in r], [p[1] for p in r]) for r in pending],
        [torch.from_numpy(r).cuda() for r in rpre],
        budget=B, eta=w.eta, max_pending_pages=w.max_pending_pages, keep_recent=w.window)
    torch.cuda.synchronize()
    kept = out["kept"].cpu().numpy()
    nk = out["n_kept"].cpu().numpy()
    for s in range(ns):
        prot_idx = O.protect_pending([p[0] for p in pending[s]], [p[1] for p in pending[s]], rpre[s], B,
                                     w.eta, w.max_pending_pages)
        prot = [pending[s][i] for i in prot_idx]
        st = O.token_states(S, retired[s], prot, w.window)
        want = O.select_tokens(score[s], st, B)
        assert nk[s] == len(want)
        np.testing.assert_array_equal(kept[s, :nk[s]], want)
        np.testing.assert_array_equal(out["pos"][s, :nk[s]].cpu().numpy(), pos_np[s, want])
        for (l, h) in [(0, 0), (17, 5), (35, 7)]:
            kin = k[s, l, h].cpu().numpy()
            vin = v[s, l, h].cpu().numpy()
            np.testing.assert_array_equal(out["k"][s, l, h, :nk[s]].view(torch.int16).cpu().numpy(), kin[want])
            np.testing.assert_array_equal(out["v"][s, l, h, :nk[s]].view(torch.int16).cpu().numpy(), vin[want])
