"""GPU parity of ckv_measure_page_effects against the fp64 oracle (Sec. 3.2).

Bar: R and R_head within 2e-3 relative (floor 1e-6) of the oracle, +inf in
the same places; window outputs, log-sum-exp and token mass to fp32/fp16
accuracy.  Every call goes through the C ABI.
"""
import numpy as np
import pytest
import torch

import oracle as O
from synth import WORKLOADS, make_layer, scaled
from tests.gpu_util import LayerOnDevice, assert_scores_close, oracle_pass

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _measure(P, ctx, dl, which, want=("R", "R_head", "o", "lse")):
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


CASES = {
    "tiny": WORKLOADS["tiny"],
    "tiny_gapped": scaled("tiny", gapped_positions=True),
    "d128_ragged": scaled("q8b", n_tokens=3000, n_q_heads=8, n_kv_heads=2, event_lo=40, event_hi=300),
    "g64_w128": scaled("q32b", n_tokens=2500, n_q_heads=8, n_kv_heads=1, window=128, event_lo=64,
                       event_hi=400),
    "w8_mha": scaled("tiny", n_tokens=1200, n_q_heads=3, n_kv_heads=3, window=8, event_lo=20,
                     event_hi=90),
    "w40_d128": scaled("q8b", n_tokens=1500, n_q_heads=6, n_kv_heads=2, window=40, page_size=24,
                       event_lo=41, event_hi=200),
    # 80-row windows: three 32-row blocks per query head, which the fast
    # token-mass kernel's whole-head workgroups do not take (general kernel,
    # separate fix-up launch)
    "w80_general": scaled("tiny", n_tokens=1700, n_q_heads=2, n_kv_heads=1, window=80, event_lo=81,
                          event_hi=300),
}


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("which", ["pre", "post"])
def test_page_effects_match_oracle(ckv, case, which):
    P, ctx = ckv
    L = make_layer(CASES[case], seed=1)
    print(f"[measure] case={case} pass={which} S={L.w.n_tokens} pages={len(L.pages)}", flush=True)
    dl = LayerOnDevice(L)
    got = _measure(P, ctx, dl, which)
    R, Rh = oracle_pass(L, which)
    assert_scores_close(got["R"], R, "R")
    assert_scores_close(got["R_head"], Rh, "R_head")
    # window outputs and lse against the oracle's full attention
    S = L.layout.s_pre if which == "pre" else L.w.n_tokens
    q = L.q_pre if which == "pre" else L.q_post
    qpos = L.qpos_pre if which == "pre" else L.qpos_post
    Ow, lse, _ = O.window_outputs(L.k[:, :S], L.v[:, :S], L.pos[:S], q, qpos)
    np.testing.assert_allclose(got["lse"], lse, rtol=0, atol=2e-4)
    scale = np.abs(Ow).max()
    np.testing.assert_allclose(got["o"], Ow, rtol=0, atol=2e-3 * scale)


def test_bruteforce_subsample_tiny(ckv):
    """The same GPU scores against the brute-force definition (masked re-run)."""
    P, ctx = ckv
    L = make_layer(WORKLOADS["tiny"], seed=2)
    dl = LayerOnDevice(L)
    got = _measure(P, ctx, dl, "post")
    sub = list(range(0, len(L.pages), 3))
    R, _ = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, [L.pages[j] for j in sub])
    assert_scores_close(got["R"][sub], R, "R (brute force)")


@pytest.mark.parametrize("case", ["d128_ragged", "g64_w128", "w8_mha", "w40_d128", "tiny_gapped", "w80_general"])
def test_token_mass(ckv, case):
    """Window mass max_h sum_p a_hpi of every token (the base score that
    fills the budget), over several head groupings and window sizes."""
    P, ctx = ckv
    L = make_layer(CASES[case], seed=3)
    print(f"[token_mass] case={case}", flush=True)
    dl = LayerOnDevice(L)
    got = _measure(P, ctx, dl, "post", want=("R", "token_mass"))
    want = O.token_mass(L.k, L.v, L.pos, L.q_post, L.qpos_post)
    np.testing.assert_allclose(got["token_mass"], want, rtol=3e-3, atol=1e-6)
    # with token mass requested the fix-up shares its launch: R still holds
    R, _ = oracle_pass(L, "post")
    assert_scores_close(got["R"], R, "R")


def test_edge_pages(ckv):
    """Hand-placed pages: a page holding every token a row sees (+inf), pages
    past every window position (0), single-token pages, a 64-token page."""
    P, ctx = ckv
    w = scaled("tiny", n_tokens=600, n_q_heads=2, n_kv_heads=1, window=4)
    L = make_layer(w, seed=4)
    L.qpos_post[:] = np.array([3, 100, 300, 599], np.int32)
    pages = [(0, 4), (4, 1), (10, 64), (200, 1), (400, 33), (560, 40)]
    L.layout.page_start = np.array([p[0] for p in pages], np.int32)
    L.layout.page_len = np.array([p[1] for p in pages], np.int32)
    dl = LayerOnDevice(L)
    got = _measure(P, ctx, dl, "post")
    R, Rh = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, pages, method="bruteforce")
    assert np.isinf(R[0])
    assert_scores_close(got["R"], R, "R")
    assert_scores_close(got["R_head"], Rh, "R_head")


def test_no_pages(ckv):
    P, ctx = ckv
    L = make_layer(WORKLOADS["tiny"], seed=5)
    dl = LayerOnDevice(L)
    kv = P.kv_view(dl.k, dl.v, dl.pos)
    win = P.window_view(dl.q_post, dl.qpos_post)
    out = P.ckv_measure_page_effects(ctx, kv, win, P.Pages([], []), want=("R", "lse"))
    torch.cuda.synchronize()
    _, lse, _ = O.window_outputs(L.k, L.v, L.pos, L.q_post, L.qpos_post)
    np.testing.assert_allclose(out["lse"].cpu().numpy(), lse, atol=2e-4, rtol=0)


def test_deterministic(ckv):
    P, ctx = ckv
    L = make_layer(WORKLOADS["tiny"], seed=6)
    dl = LayerOnDevice(L)
    a = _measure(P, ctx, dl, "post")
    b = _measure(P, ctx, dl, "post")
    assert np.array_equal(a["R"], b["R"]) and np.array_equal(a["o"], b["o"])


@pytest.mark.parametrize("mass", [False, True])
@pytest.mark.parametrize("which", ["single_heavy", "two_heavy_straddling"])
def test_dominant_page(ckv, which, mass):
    """Pages that hold nearly all of a row's attention mass (A -> 1): the
    closed form of Eq. (6) cancels there; the library recomputes such rows
    without the page and must still meet the score tolerance.  With token
    mass requested the recomputation runs inside the token-mass launch."""
    P, ctx = ckv
    w = scaled("tiny", n_tokens=2048, n_q_heads=4, n_kv_heads=1)
    L = make_layer(w, seed=7)
    from synth import bf16_bits, bf16_bits_to_f32
    k = bf16_bits_to_f32(L.k).copy()
    q = bf16_bits_to_f32(L.q_post)
    qdir = q[:, :, :].mean(axis=(0, 1))
    qdir /= np.linalg.norm(qdir)
    if which == "single_heavy":
        st = int(L.layout.page_start[len(L.pages) // 2])
        k[0, st + 3] = qdir * 60.0          # logit ~ 60/8 * |q| per row: dominant
    else:
        # page straddling a 64-token boundary, two heavy tokens inside it
        j = int(np.argmin(np.abs((L.layout.page_start % 64) - 56)))
        st = int(L.layout.page_start[j])
        k[0, st + 2] = qdir * 55.0
        k[0, st + 9] = qdir * 52.0
    L.k = bf16_bits(k)
    dl = LayerOnDevice(L)
    got = _measure(P, ctx, dl, "post", want=("R", "R_head") + (("token_mass",) if mass else ()))
    R, Rh = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, method="closed")
    if mass:
        np.testing.assert_allclose(got["token_mass"], O.token_mass(L.k, L.v, L.pos, L.q_post, L.qpos_post),
                                   rtol=3e-3, atol=1e-6)
    # the oracle confirms the page is dominant for some rows
    import math
    K, V, Q = O.as_f64(L.k), O.as_f64(L.v), O.as_f64(L.q_post)
    s = O.head_logits(Q[0], K[0], 1 / math.sqrt(64))
    a, _ = O.attend(s, O.visibility(L.pos, L.qpos_post), V[0])
    page = [p for p in L.pages if p[0] <= st < p[0] + p[1]][0]
    A = a[:, page[0]:page[0] + page[1]].sum(1)
    assert A.max() > 0.999
    assert_scores_close(got["R"], R, "R")
    assert_scores_close(got["R_head"], Rh, "R_head")


@pytest.mark.parametrize("which", ["max_inside", "max_outside", "max_second_tile", "max_first_part_g32",
                                   "max_first_part_g64", "max_second_part_g64", "max_after_page_g64",
                                   "max_near_page_g32"])
def test_heavy_page_band(ckv, which):
    """Pages carrying between 0.9 and 0.99 of a row's mass.  A page that holds
    its row's largest logit inside one 64-token tile keeps the closed form of
    Eq. (6) up to A = 0.99 (its float16 weights are the ones that formed o),
    and so does one that crosses into the next tile of the same window-pass
    split with that logit before the crossing (max_first_part: 32- and
    64-token pages over 128-token splits, so every other tile boundary is
    also a split boundary, where the page is recomputed).  A page whose
    tokens share the mass while a token outside it holds the row's largest
    logit, and a page that straddles a 64-token boundary with its largest
    logit after it (the window pass weighted its first part against an older
    reference; max_second_tile over one-tile splits, max_second_part over
    128-token splits), are listed above A = 0.8: recomputed by definition,
    or, where the page lies in the tile before the one where the logit
    entered the split's reference or in a later tile of that split, evaluated
    with the window pass's own weights (max_second_part; max_after_page,
    whose largest logit is the token just after a page that carries the
    mass; max_near_page, a page inside one tile with the largest logit in
    the split's other tile).  All must meet the tolerance."""
    P, ctx = ckv
    import math
    split128 = which[:-4] in ("max_first_part", "max_second_part", "max_after_page", "max_near_page")
    if split128:
        # 8 KV heads over 4096 tokens: 32 splits of 128 tokens
        w = scaled("tiny", n_tokens=4096, n_q_heads=16, n_kv_heads=8, page_size=int(which[-2:]))
    else:
        w = scaled("tiny", n_tokens=2048, n_q_heads=4, n_kv_heads=1)
    L = make_layer(w, seed=11)
    from synth import bf16_bits, bf16_bits_to_f32
    k = bf16_bits_to_f32(L.k).copy()
    q = bf16_bits_to_f32(L.q_post)
    qdir = q.mean(axis=(0, 1))
    qdir /= np.linalg.norm(qdir)
    starts, lens = L.layout.page_start, L.layout.page_len
    full = np.flatnonzero(lens == lens.max())
    ends = starts + lens - 1
    if which == "max_after_page_g64":
        # every token of a page across a tile boundary at one logit for one
        # row of the group's first query head (a ladder over the pages), the
        # token just after the page (in the page's second tile) one higher
        strad = np.flatnonzero((starts // 64 != ends // 64) & (ends + 1 < w.n_tokens))[::2]   # apart
        logit = np.linspace(8.0, 16.0, len(strad))
        group = w.n_q_heads // w.n_kv_heads
        for n, j in enumerate(strad):
            for g in range(w.n_kv_heads):
                qr = q[g * group, (n + 7 * g) % w.window]
                c = logit[(n + 5 * g) % len(strad)] * math.sqrt(w.head_dim) / float(qr @ qr)
                k[g, int(starts[j]):int(ends[j]) + 1] = qr * c
                k[g, int(ends[j]) + 1] = qr * (c * (1.0 + 1.0 / logit[(n + 5 * g) % len(strad)]))
        probe = strad
    elif which == "max_near_page_g32":
        # one page inside one tile per 128-token split (the split's first
        # tile in even splits, its second in odd ones), every token at one
        # logit for one row of the group's first query head (a ladder over
        # the pages), and the first token of the split's other tile one higher
        inner = np.flatnonzero(starts // 64 == ends // 64)
        probe = []
        for sp in range(w.n_tokens // 128):
            pick = [j for j in inner if starts[j] // 128 == sp and (starts[j] // 64) % 2 == sp % 2]
            if pick and ends[pick[0]] < w.n_tokens - 1:
                probe.append(pick[0])
        logit = np.linspace(8.0, 16.0, len(probe))
        group = w.n_q_heads // w.n_kv_heads
        for n, j in enumerate(probe):
            t = int(starts[j]) // 64
            other = (t + 1) * 64 if t % 2 == 0 else (t - 1) * 64
            for g in range(w.n_kv_heads):
                qr = q[g * group, (n + 7 * g) % w.window]
                lg = logit[(n + 5 * g) % len(probe)]
                c = lg * math.sqrt(w.head_dim) / float(qr @ qr)
                k[g, int(starts[j]):int(ends[j]) + 1] = qr * c
                k[g, other] = qr * (c * (1.0 + 1.0 / lg))
    elif split128:
        # every page across a tile boundary gets a heavy token in each KV
        # head, its first one (before the boundary) or the first after the
        # boundary, aimed at one row of the group's first query head with a
        # logit from a ladder that puts A on both sides of 0.9 and 0.99
        strad = np.flatnonzero(starts // 64 != ends // 64)
        logit = np.linspace(9.0, 16.0, len(strad))
        group = w.n_q_heads // w.n_kv_heads
        for n, j in enumerate(strad):
            for g in range(w.n_kv_heads):
                qr = q[g * group, (n + 7 * g) % w.window]
                at = int(starts[j]) if which.startswith("max_first") else (int(starts[j]) // 64 + 1) * 64
                k[g, at] = qr * (logit[(n + 5 * g) % len(strad)] * math.sqrt(w.head_dim) / float(qr @ qr))
        probe = strad
    elif which == "max_inside":
        # one heavy token per page, at strengths that put A on both sides of
        # 0.9 and 0.99 across the rows
        strengths = np.geomspace(30.0, 200.0, 24)
        picks = full[np.linspace(0, len(full) - 1, len(strengths)).astype(int)]
        for j, c in zip(picks, strengths):
            k[0, int(starts[j]) + 1] = qdir * c
        probe = picks
    elif which == "max_second_tile":
        strad = np.flatnonzero(starts // 64 != ends // 64)
        strengths = np.geomspace(30.0, 200.0, min(24, len(strad)))
        picks = strad[np.linspace(0, len(strad) - 1, len(strengths)).astype(int)]
        for j, c in zip(picks, strengths):
            k[0, (int(starts[j]) // 64 + 1) * 64] = qdir * c    # first token after the boundary
        probe = picks
    else:
        # every token of one page equally strong, one token elsewhere a little
        # stronger: the page carries most of the mass without the largest logit
        j = int(full[len(full) // 2])
        st, ln = int(starts[j]), int(lens[j])
        k[0, st:st + ln] = qdir * 80.0
        k[0, int(starts[full[1]]) + 2] = qdir * 82.0
        probe = [j]
    L.k = bf16_bits(k)
    dl = LayerOnDevice(L)
    got = _measure(P, ctx, dl, "post")
    R, Rh = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, method="closed")
    K, V, Q = O.as_f64(L.k), O.as_f64(L.v), O.as_f64(L.q_post)
    vis = O.visibility(L.pos, L.qpos_post)
    band = inside = 0
    group = Q.shape[0] // K.shape[0]
    for h in range(Q.shape[0]):
        s = O.head_logits(Q[h], K[h // group], 1 / math.sqrt(K.shape[2]))
        a, _ = O.attend(s, vis, V[h // group])
        for j in probe:
            st, ln = int(starts[j]), int(lens[j])
            A = a[:, st:st + ln].sum(1)
            sel = (A > 0.9) & (A < 0.99)
            band += int(sel.sum())
            if split128 and (st // 64 + 1) % 2 == 1:
                # a tile boundary inside a split (max_first_part: the closed
                # form is kept), or a page in the split's first tile
                # (max_near_page: weighted against the older reference)
                inside += int(sel.sum())
            if which == "max_outside" and sel.any():
                # the row's largest logit lies outside the page
                sm = np.where(vis, s, -np.inf)
                assert (sm[sel, st:st + ln].max(1) < sm[sel].max(1)).all()
    print(f"[measure] {which}: {band} (page, row) pairs with 0.9 < A < 0.99, {inside} of them across a "
          f"tile boundary inside a split", flush=True)
    assert band >= 20
    if split128:
        assert inside >= 10 and band - inside >= 10
    assert_scores_close(got["R"], R, "R")
    assert_scores_close(got["R_head"], Rh, "R_head")


def test_batch_matches_single_calls(ckv):
    """ckv_measure_page_effects_batch over problems of different shapes (head
    width, grouping, window, prefix) gives, problem by problem, exactly what
    the single call gives."""
    P, ctx = ckv
    probs = []
    for case, which in (("tiny", "pre"), ("tiny", "post"), ("d128_ragged", "post"), ("w8_mha", "pre")):
        L = make_layer(CASES[case], seed=21)
        dl = LayerOnDevice(L)
        if which == "pre":
            kv = P.kv_view(dl.k, dl.v, dl.pos, n_tokens=L.layout.s_pre)
            win = P.window_view(dl.q_pre, dl.qpos_pre)
        else:
            kv = P.kv_view(dl.k, dl.v, dl.pos)
            win = P.window_view(dl.q_post, dl.qpos_post)
        probs.append((kv, win, P.Pages(L.layout.page_start, L.layout.page_len), dl))
    want = ("R", "R_head", "o", "lse", "token_mass")
    batch = P.ckv_measure_page_effects_batch(ctx, [p[0] for p in probs], [p[1] for p in probs],
                                             [p[2] for p in probs], want=want)
    single = [P.ckv_measure_page_effects(ctx, kv, win, pg, want=want) for kv, win, pg, _ in probs]
    torch.cuda.synchronize()
    for b, s in zip(batch, single):
        for k in want:
            assert np.array_equal(b[k].cpu().numpy().view(np.uint32), s[k].cpu().numpy().view(np.uint32)), k
    # a bad problem is reported before anything runs
    bad = P.Pages([0], [65])
    with pytest.raises(P.CKVError) as e:
        P.ckv_measure_page_effects_batch(ctx, [probs[0][0], probs[1][0]], [probs[0][1], probs[1][1]],
                                         [probs[0][2], bad])
    assert e.value.code == -2 and "problem 1" in str(e.value)
