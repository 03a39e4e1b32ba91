"""GPU parity of ckv_measure_recorded: page deletion effects from recorded
window outputs (Sec. 3.2: the engine records the window's attention outputs
during the forward pass), against the fp64 oracle.

The recorded o and log-sum-exp are the oracle's own, rounded to float32 (an
exact engine), or the library's outputs from ckv_measure_page_effects.  Bar:
R and R_head within 2e-3 relative, +inf in the same places; for pages that
carry between 0.5 and 0.99 of a row's mass the documented bound adds a few
ulp(lse) / (1 - A) (the recorded lse and the page's float32 logits fix 1 - A
to that accuracy); token mass within 3e-3.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
from synth import WORKLOADS, bf16_bits, bf16_bits_to_f32, make_layer, scaled
from tests.gpu_util import REL_TOL, LayerOnDevice

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _views(P, dl, which):
    L = dl.L
    if which == "pre":
        return (P.kv_view(dl.k, dl.v, dl.pos, n_tokens=L.layout.s_pre), P.window_view(dl.q_pre, dl.qpos_pre))
    return P.kv_view(dl.k, dl.v, dl.pos), P.window_view(dl.q_post, dl.qpos_post)


def _oracle_outputs(L, which, heads=None):
    S = L.layout.s_pre if which == "pre" else L.w.n_tokens
    q = L.q_pre if which == "pre" else L.q_post
    qpos = L.qpos_pre if which == "pre" else L.qpos_post
    O_, lse, _ = O.window_outputs(L.k[:, :S], L.v[:, :S], L.pos[:S], q, qpos)
    return O_, lse


def _recorded(P, ctx, dl, which, o, lse, want=("R", "R_head")):
    kv, win = _views(P, dl, which)
    pages = P.Pages(dl.L.layout.page_start, dl.L.layout.page_len)
    out = P.ckv_measure_recorded(ctx, kv, win, pages, torch.from_numpy(np.ascontiguousarray(o, np.float32)).cuda(),
                                 torch.from_numpy(np.ascontiguousarray(lse, np.float32)).cuda(), want=want)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if torch.is_tensor(v) else v) for k, v in out.items()}


def _allowance(L, which, lse, heads=None):
    """Per (page, query head) relative tolerance: the score tolerance, plus,
    for rows where the page carries between half and 0.99 of the mass (those
    the library evaluates from the page's own tokens against the recorded
    lse), 4 ulp(lse) / (1 - A): the recorded lse and the page's float32
    logits fix 1 - A only to a few ulp of lse.  Above 0.99 the output without
    the page is recomputed from the rest of the row, with no extra allowance."""
    S = L.layout.s_pre if which == "pre" else L.w.n_tokens
    q = L.q_pre if which == "pre" else L.q_post
    qpos = L.qpos_pre if which == "pre" else L.qpos_post
    K, V, Q = O.as_f64(L.k[:, :S]), O.as_f64(L.v[:, :S]), O.as_f64(q)
    vis = O.visibility(L.pos[:S], qpos)
    group = Q.shape[0] // K.shape[0]
    tol = np.full((len(L.pages), Q.shape[0]), REL_TOL)
    amax = 0.0
    for h in (range(Q.shape[0]) if heads is None else heads):
        s = O.head_logits(Q[h], K[h // group], 1 / math.sqrt(K.shape[2]))
        a, _ = O.attend(s, vis, V[h // group])
        with np.errstate(invalid="ignore"):
            ulp = np.spacing(np.abs(np.asarray(lse[h], np.float32))).astype(np.float64)
        for j, (s0, ln) in enumerate(L.pages):
            A = a[:, s0:s0 + ln].sum(1)
            amax = max(amax, float(A.max()) if A.size else 0.0)
            big = (A > 0.5) & (A <= 0.99)    # above 0.99 the complement pass is exact
            if big.any():
                tol[j, h] += float(np.max(4 * ulp[big] / (1 - np.minimum(A[big], 1 - 1e-12))))
    return tol, amax


def _assert_within(got, want, tol, what):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    assert np.array_equal(np.isinf(got), np.isinf(want)), f"{what}: inf mismatch"
    fin = np.isfinite(want)
    rel = np.abs(got[fin] - want[fin]) / np.maximum(want[fin], 1e-6)
    lim = np.broadcast_to(tol, want.shape)[fin]
    print(f"[parity] {what}: worst relative error {rel.max() if rel.size else 0:.3g}, "
          f"worst error/allowance {np.max(rel / lim) if rel.size else 0:.3g}", flush=True)
    bad = np.flatnonzero(rel > lim)
    assert bad.size == 0, f"{what}: {bad.size} values outside the allowance, worst rel {rel.max():.3g}"


CASES = {
    "tiny": WORKLOADS["tiny"],
    "tiny_gapped": scaled("tiny", gapped_positions=True),
    "d128_ragged": scaled("q8b", n_tokens=3000, n_q_heads=8, n_kv_heads=2, window=40),
    "w8_mha": scaled("tiny", n_tokens=1500, n_q_heads=2, n_kv_heads=2, window=8),
}


@pytest.mark.parametrize("which", ["pre", "post"])
@pytest.mark.parametrize("case", list(CASES))
def test_recorded_exact_outputs(ckv, case, which):
    P, ctx = ckv
    L = make_layer(CASES[case], seed=12)
    print(f"[recorded] case={case} {which}", flush=True)
    dl = LayerOnDevice(L)
    o, lse = _oracle_outputs(L, which)
    got = _recorded(P, ctx, dl, which, o, lse)
    S = L.layout.s_pre if which == "pre" else L.w.n_tokens
    q = L.q_pre if which == "pre" else L.q_post
    qpos = L.qpos_pre if which == "pre" else L.qpos_post
    method = "bruteforce" if L.w.n_tokens <= 2048 else "closed"
    R, Rh = O.page_effects(L.k[:, :S], L.v[:, :S], L.pos[:S], q, qpos, L.pages, method=method)
    tol, _ = _allowance(L, which, lse)
    _assert_within(got["R"], R, tol.max(axis=1), "R")
    _assert_within(got["R_head"], Rh, tol, "R_head")


def test_recorded_from_library_outputs(ckv):
    """The outputs ckv_measure_page_effects returns, fed back as recorded
    ones, give effects within the score tolerance of the oracle."""
    P, ctx = ckv
    L = make_layer(scaled("q8b", n_tokens=6000, n_q_heads=8, n_kv_heads=2), seed=13)
    dl = LayerOnDevice(L)
    kv, win = _views(P, dl, "post")
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    full = P.ckv_measure_page_effects(ctx, kv, win, pages, want=("R", "R_head", "o", "lse"))
    rec = P.ckv_measure_recorded(ctx, kv, win, pages, full["o"].contiguous(), full["lse"].contiguous(),
                                 want=("R", "R_head", "token_mass"))
    torch.cuda.synchronize()
    R, Rh = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, method="closed")
    tol, _ = _allowance(L, "post", full["lse"].cpu().numpy())
    _assert_within(rec["R"].cpu().numpy(), R, tol.max(axis=1), "R")
    _assert_within(rec["R_head"].cpu().numpy(), Rh, tol, "R_head")
    tm = O.token_mass(L.k, L.v, L.pos, L.q_post, L.qpos_post)
    np.testing.assert_allclose(rec["token_mass"].cpu().numpy(), tm, rtol=3e-3, atol=1e-6)


def test_recorded_edge_pages(ckv):
    """A page holding every token a row sees (+inf), pages past every window
    position (0), single-token and 64-token pages."""
    P, ctx = ckv
    w = scaled("tiny", n_tokens=600, n_q_heads=2, n_kv_heads=1, window=4)
    L = make_layer(w, seed=4)
    L.qpos_post[:] = np.array([3, 100, 300, 599], np.int32)
    pages = [(0, 4), (4, 1), (10, 64), (200, 1), (400, 33), (560, 40)]
    L.layout.page_start = np.array([p[0] for p in pages], np.int32)
    L.layout.page_len = np.array([p[1] for p in pages], np.int32)
    dl = LayerOnDevice(L)
    o, lse = _oracle_outputs(L, "post")
    got = _recorded(P, ctx, dl, "post", o, lse)
    R, Rh = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, pages, method="bruteforce")
    assert np.isinf(R[0])
    tol, _ = _allowance(L, "post", lse)
    _assert_within(got["R"], R, tol.max(axis=1), "R")
    _assert_within(got["R_head"], Rh, tol, "R_head")


@pytest.mark.parametrize("which", ["single_heavy", "two_heavy_straddling"])
def test_recorded_dominant_page(ckv, which):
    """Pages with A -> 1 go through the recorded fix-up: within the score
    tolerance plus the documented bound."""
    P, ctx = ckv
    w = scaled("tiny", n_tokens=2048, n_q_heads=4, n_kv_heads=1)
    L = make_layer(w, seed=7)
    k = bf16_bits_to_f32(L.k).copy()
    q = bf16_bits_to_f32(L.q_post)
    qdir = q.mean(axis=(0, 1))
    qdir /= np.linalg.norm(qdir)
    if which == "single_heavy":
        st = int(L.layout.page_start[len(L.pages) // 2])
        k[0, st + 3] = qdir * 60.0
    else:
        j = int(np.argmin(np.abs((L.layout.page_start % 64) - 56)))
        st = int(L.layout.page_start[j])
        k[0, st + 2] = qdir * 55.0
        k[0, st + 9] = qdir * 52.0
    L.k = bf16_bits(k)
    dl = LayerOnDevice(L)
    o, lse = _oracle_outputs(L, "post")
    got = _recorded(P, ctx, dl, "post", o, lse)
    R, Rh = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, method="closed")
    tol, amax = _allowance(L, "post", lse)
    assert amax > 0.999
    _assert_within(got["R_head"], Rh, tol, f"R_head dominant {which}")


def test_recorded_q8b_sampled_heads(ckv):
    """Full-size layer in the benchmark's configuration, recorded outputs from
    the library: per-head effects of every page for sampled heads."""
    P, ctx = ckv
    L = make_layer(WORKLOADS["q8b"], seed=0)
    dl = LayerOnDevice(L)
    kv, win = _views(P, dl, "post")
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    full = P.ckv_measure_page_effects(ctx, kv, win, pages, want=("R", "o", "lse"))
    rec = P.ckv_measure_recorded(ctx, kv, win, pages, full["o"].contiguous(), full["lse"].contiguous(),
                                 want=("R", "R_head"))
    torch.cuda.synchronize()
    heads = [0, 17, 31]
    _, Rh = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, method="closed", heads=heads)
    got = rec["R_head"].cpu().numpy()
    tol, _ = _allowance(L, "post", full["lse"].cpu().numpy(), heads)
    for h in heads:
        _assert_within(got[:, h], Rh[:, h], tol[:, h], f"R_head[:, {h}]")
    assert np.all(rec["R"].cpu().numpy() >= got.max(axis=1) * (1 - 1e-7))


def test_recorded_argument_errors(ckv):
    P, ctx = ckv
    L = make_layer(WORKLOADS["tiny"], seed=1)
    dl = LayerOnDevice(L)
    kv, win = _views(P, dl, "post")
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    o = torch.zeros(L.w.n_q_heads * L.w.window * L.w.head_dim + 1, dtype=torch.float32, device="cuda")
    lse = torch.zeros(L.w.n_q_heads * L.w.window, dtype=torch.float32, device="cuda")
    with pytest.raises(P.CKVError) as e:          # misaligned recorded outputs
        P.ckv_measure_recorded(ctx, kv, win, pages, o[1:], lse)
    assert e.value.code == -1


def test_recorded_many_dominant_pairs(ckv):
    """1280 window rows (32 query heads x 40 rows over 4 KV heads), each with
    a page that carries > 0.99 of its mass: every (page, row) pair goes
    through the complement pass (more pairs than the pass's 1024-pair
    chunk), and R, R_head match the fp64 oracle at 2e-3."""
    P, ctx = ckv
    rng = np.random.default_rng(44)
    S, d, Hq, Hkv, W = 2048, 128, 32, 4, 40
    u = rng.standard_normal(d)
    q = bf16_bits((u + 0.3 * rng.standard_normal((Hq, W, d))).astype(np.float32))
    k = rng.standard_normal((Hkv, S, d))
    pages = [(512 + 32 * i, 32) for i in range(32)]
    dom = [3 + 5 * g for g in range(Hkv)]
    for g, j in enumerate(dom):
        st = pages[j][0]
        k[g, st:st + 32] = u + 0.05 * rng.standard_normal((32, d))
    v = rng.standard_normal((Hkv, S, d))
    kb, vb = bf16_bits(k.astype(np.float32)), bf16_bits(v.astype(np.float32))
    pos = np.arange(S, dtype=np.int32)
    qpos = np.arange(S, S + W, dtype=np.int32)
    o, lse, _ = O.window_outputs(kb, vb, pos, q, qpos)
    # every row's dominant page holds > 0.99 of the mass (oracle, fp64)
    K, V, Q = O.as_f64(kb), O.as_f64(vb), O.as_f64(q)
    vis = O.visibility(pos, qpos)
    amin = 1.0
    for h in range(Hq):
        g = h // (Hq // Hkv)
        a, _ = O.attend(O.head_logits(Q[h], K[g], 1 / np.sqrt(d)), vis, V[g])
        st = pages[dom[g]][0]
        amin = min(amin, float(a[:, st:st + 32].sum(1).min()))
    print(f"[recorded] many dominant pairs: {Hq * W} rows, smallest dominant mass {amin:.5f}", flush=True)
    assert amin > 0.99
    from tests.gpu_util import dev_bf16, dev_i32, assert_scores_close
    kv = P.kv_view(dev_bf16(kb), dev_bf16(vb), dev_i32(pos))
    win = P.window_view(dev_bf16(q), dev_i32(qpos))
    pl = P.Pages([p[0] for p in pages], [p[1] for p in pages])
    out = P.ckv_measure_recorded(ctx, kv, win, pl, torch.from_numpy(np.ascontiguousarray(o, np.float32)).cuda(),
                                 torch.from_numpy(np.ascontiguousarray(lse, np.float32)).cuda(),
                                 want=("R", "R_head"))
    torch.cuda.synchronize()
    R, Rh = O.page_effects(kb, vb, pos, q, qpos, pages, method="closed")
    assert_scores_close(out["R"].cpu().numpy(), R, "R (many dominant pairs)")
    assert_scores_close(out["R_head"].cpu().numpy().reshape(Rh.shape), Rh, "R_head (many dominant pairs)")
