"""Paged caches (ckv_kv_view.slot): every call on a pool whose rows hold the
tokens in a scattered order must give results bit-identical to the same call
on the contiguous cache (the kernels run the same arithmetic; only the row
addresses change), and selection without compaction (out = NULL) must pick
the same index set as the compacting call.

The contiguous results are themselves checked against the fp64 oracle by the
other GPU tests.
"""
import numpy as np
import pytest
import torch

from synth import WORKLOADS, bf16_bits, make_layer, make_scores, scaled
from tests.gpu_util import LayerOnDevice, dev_bf16, dev_i32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _pool(L, seed, extra=0.5):
    """Scatter the layer's tokens over a pool of about (1 + extra) S rows;
    the other rows hold unrelated finite values."""
    rng = np.random.default_rng(seed)
    Hkv, S, d = L.k.shape
    rows = S + int(extra * S) + 7
    slot = rng.choice(rows, S, replace=False).astype(np.int32)
    kp = bf16_bits(rng.standard_normal((Hkv, rows, d), dtype=np.float32))
    vp = bf16_bits(rng.standard_normal((Hkv, rows, d), dtype=np.float32))
    kp[:, slot] = L.k
    vp[:, slot] = L.v
    return dev_bf16(kp), dev_bf16(vp), slot


def _both(P, dl, kp, vp, slot, which):
    L = dl.L
    n = L.layout.s_pre if which == "pre" else L.w.n_tokens
    q, qp = (dl.q_pre, dl.qpos_pre) if which == "pre" else (dl.q_post, dl.qpos_post)
    dense = P.kv_view(dl.k, dl.v, dl.pos, n_tokens=n)
    paged = P.kv_view(kp, vp, dl.pos, n_tokens=n, slot=dev_i32(slot[:n]))
    return dense, paged, P.window_view(q, qp)


def _same(a, b, what):
    a, b = a.cpu().numpy(), b.cpu().numpy()
    assert a.shape == b.shape
    assert np.array_equal(a.view(np.uint32) if a.dtype == np.float32 else a,
                          b.view(np.uint32) if b.dtype == np.float32 else b), what


CASES = {
    "tiny": WORKLOADS["tiny"],
    "d128_ragged": scaled("q8b", n_tokens=3000, n_q_heads=8, n_kv_heads=2, window=40),
    "w8_gqa5": scaled("q8b", n_tokens=2500, n_q_heads=10, n_kv_heads=2, window=8, page_size=16),
}


@pytest.mark.parametrize("which", ["pre", "post"])
@pytest.mark.parametrize("case", list(CASES))
def test_measure_bit_identical(ckv, case, which):
    P, ctx = ckv
    L = make_layer(CASES[case], seed=31)
    print(f"[paged] measure case={case} {which}", flush=True)
    dl = LayerOnDevice(L)
    kp, vp, slot = _pool(L, seed=1)
    dense, paged, win = _both(P, dl, kp, vp, slot, which)
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    want = ("R", "R_head", "o", "lse", "token_mass")
    a = P.ckv_measure_page_effects(ctx, dense, win, pages, want=want)
    b = P.ckv_measure_page_effects(ctx, paged, win, pages, want=want)
    torch.cuda.synchronize()
    for k in want:
        _same(a[k], b[k], k)
    # recorded outputs over the pool
    ra = P.ckv_measure_recorded(ctx, dense, win, pages, a["o"].contiguous(), a["lse"].contiguous(),
                                want=("R", "R_head", "token_mass"))
    rb = P.ckv_measure_recorded(ctx, paged, win, pages, a["o"].contiguous(), a["lse"].contiguous(),
                                want=("R", "R_head", "token_mass"))
    torch.cuda.synchronize()
    for k in ("R", "R_head", "token_mass"):
        _same(ra[k], rb[k], "recorded " + k)


def test_dominant_page_fixups_bit_identical(ckv):
    """A page that carries nearly all of some rows' mass: the fix-up kernels
    (window-pass splits, recorded page-only and complement passes) read the
    pool too."""
    P, ctx = ckv
    from synth import bf16_bits_to_f32
    L = make_layer(scaled("tiny", n_tokens=2048, n_q_heads=4, n_kv_heads=1), seed=7)
    k = bf16_bits_to_f32(L.k).copy()
    qdir = bf16_bits_to_f32(L.q_post).mean(axis=(0, 1))
    qdir /= np.linalg.norm(qdir)
    st = int(L.layout.page_start[len(L.pages) // 2])
    k[0, st + 3] = qdir * 60.0
    L.k = bf16_bits(k)
    dl = LayerOnDevice(L)
    kp, vp, slot = _pool(L, seed=2)
    dense, paged, win = _both(P, dl, kp, vp, slot, "post")
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    a = P.ckv_measure_page_effects(ctx, dense, win, pages, want=("R", "R_head", "o", "lse"))
    b = P.ckv_measure_page_effects(ctx, paged, win, pages, want=("R", "R_head", "o", "lse"))
    ra = P.ckv_measure_recorded(ctx, dense, win, pages, a["o"].contiguous(), a["lse"].contiguous(),
                                want=("R", "R_head"))
    rb = P.ckv_measure_recorded(ctx, paged, win, pages, a["o"].contiguous(), a["lse"].contiguous(),
                                want=("R", "R_head"))
    torch.cuda.synchronize()
    for k_ in ("R", "R_head"):
        _same(a[k_], b[k_], k_)
        _same(ra[k_], rb[k_], "recorded " + k_)


def test_window_weight_fixups_bit_identical(ckv):
    """Pages inside one tile of a 128-token window-pass split carrying most of
    a row's mass while the row's largest logit lies in the split's other
    tile: the fix-up evaluates them with the window pass's own weights, and
    through the pool it must give the same bits."""
    P, ctx = ckv
    import math
    from synth import bf16_bits_to_f32
    w = scaled("tiny", n_tokens=4096, n_q_heads=16, n_kv_heads=8, page_size=32)
    L = make_layer(w, seed=11)
    k = bf16_bits_to_f32(L.k).copy()
    q = bf16_bits_to_f32(L.q_post)
    starts, ends = L.layout.page_start, L.layout.page_start + L.layout.page_len - 1
    inner = [j for j in np.flatnonzero(starts // 64 == ends // 64) if ends[j] < w.n_tokens - 1]
    probe = [next(j for j in inner if starts[j] // 128 == sp and (starts[j] // 64) % 2 == sp % 2)
             for sp in range(w.n_tokens // 128)
             if any(starts[j] // 128 == sp and (starts[j] // 64) % 2 == sp % 2 for j in inner)]
    group = w.n_q_heads // w.n_kv_heads
    for n, j in enumerate(probe):
        t = int(starts[j]) // 64
        other = (t + 1) * 64 if t % 2 == 0 else (t - 1) * 64
        for g in range(w.n_kv_heads):
            qr = q[g * group, (n + 7 * g) % w.window]
            lg = 8.0 + 8.0 * ((n + 5 * g) % len(probe)) / max(len(probe) - 1, 1)
            c = lg * math.sqrt(w.head_dim) / float(qr @ qr)
            k[g, int(starts[j]):int(ends[j]) + 1] = qr * c
            k[g, other] = qr * (c * (1.0 + 1.0 / lg))
    L.k = bf16_bits(k)
    dl = LayerOnDevice(L)
    kp, vp, slot = _pool(L, seed=5)
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    for which in ("pre", "post"):
        dense, paged, win = _both(P, dl, kp, vp, slot, which)
        a = P.ckv_measure_page_effects(ctx, dense, win, pages, want=("R", "R_head"))
        b = P.ckv_measure_page_effects(ctx, paged, win, pages, want=("R", "R_head"))
        torch.cuda.synchronize()
        for k_ in ("R", "R_head"):
            _same(a[k_], b[k_], which + " " + k_)


def test_joint_bit_identical(ckv):
    P, ctx = ckv
    w = scaled("stress", n_tokens=4096, n_q_heads=8, n_kv_heads=2, max_cand=64)
    L = make_layer(w, seed=5)
    dl = LayerOnDevice(L)
    kp, vp, slot = _pool(L, seed=3)
    dense, paged, win = _both(P, dl, kp, vp, slot, "post")
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    outs = []
    for kv in (dense, paged):
        m = P.ckv_measure_page_effects(ctx, kv, win, pages, want=("R", "o", "lse"))
        cl = P.ckv_classify_pages(ctx, torch.zeros_like(m["R"]), m["R"],
                                  force=torch.tensor(L.forced.astype(np.uint8)).cuda(), max_cand=64)
        jt = P.ckv_joint_test(ctx, kv, win, m["o"], m["lse"], pages, cl["cand"], cl["n_cand"], 64, 0.01)
        outs.append(jt)
    torch.cuda.synchronize()
    _same(outs[0]["accepted"], outs[1]["accepted"], "accepted")
    _same(outs[0]["union_R"], outs[1]["union_R"], "union_R")
    assert int(outs[0]["n_accepted"].item()) > 0


def test_out_of_range_slots_are_clamped(ckv):
    """Slots outside the pool read its last row (in bounds): the same as a
    contiguous cache holding the last row's values at those tokens."""
    P, ctx = ckv
    L = make_layer(WORKLOADS["tiny"], seed=8)
    dl = LayerOnDevice(L)
    kp, vp, slot = _pool(L, seed=4)
    rows = kp.shape[1]
    slot = slot.copy()
    slot[5], slot[900] = rows + 100, -3
    kd, vd = L.k.copy(), L.v.copy()
    last_k = kp[:, rows - 1].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    last_v = vp[:, rows - 1].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    kd[:, [5, 900]] = last_k[:, None]
    vd[:, [5, 900]] = last_v[:, None]
    dense = P.kv_view(dev_bf16(kd), dev_bf16(vd), dl.pos)
    paged = P.kv_view(kp, vp, dl.pos, slot=dev_i32(slot))
    win = P.window_view(dl.q_post, dl.qpos_post)
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    a = P.ckv_measure_page_effects(ctx, dense, win, pages, want=("R", "token_mass"))
    b = P.ckv_measure_page_effects(ctx, paged, win, pages, want=("R", "token_mass"))
    torch.cuda.synchronize()
    _same(a["R"], b["R"], "R")
    _same(a["token_mass"], b["token_mass"], "token_mass")


def test_selection_without_compaction(ckv):
    """out = NULL: the same kept indices, nothing copied."""
    P, ctx = ckv
    n_seq, L_, H, d, cap = 2, 2, 2, 64, 3000
    k = torch.randint(-32768, 32767, (n_seq, L_, H, cap, d), dtype=torch.int16).view(torch.bfloat16).cuda()
    v = torch.randint(-32768, 32767, (n_seq, L_, H, cap, d), dtype=torch.int16).view(torch.bfloat16).cuda()
    pos = torch.arange(cap, dtype=torch.int32).repeat(n_seq, 1).cuda()
    score = torch.from_numpy(np.stack([make_scores(cap, seed=s) for s in range(n_seq)])).cuda()
    nt = [3000, 2100]
    pend = [P.Pages([100, 200], [16, 16]), P.Pages([50], [8])]
    rpre = [torch.tensor([0.5, 0.7], device="cuda"), torch.tensor([0.2], device="cuda")]
    ret = [P.Pages([300], [32]), P.Pages([], [])]
    full = P.ckv_select_and_compact(ctx, k, v, pos, nt, score, ret, pend, rpre, budget=700)
    only = P.ckv_select_and_compact(ctx, k, v, pos, nt, score, ret, pend, rpre, budget=700, compact=False)
    torch.cuda.synchronize()
    _same(full["kept"], only["kept"], "kept")
    _same(full["n_kept"], only["n_kept"], "n_kept")
    assert only["k"] is None
