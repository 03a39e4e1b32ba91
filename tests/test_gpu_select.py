"""GPU parity of ckv_select_and_compact (Sec. 3.3, Eq. (12)-(13); Sec. 3.1, Eq. (4)).

Bit-exact bar: given the same float32 scores, pending effects and page lists,
the kept index set must equal the oracle's, and the compacted K, V and
positions must equal fancy indexing of the inputs byte for byte.
"""
import numpy as np
import pytest
import torch

import oracle as O
from synth import make_scores

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _pages(rng, S, n, maxlen=64):
    starts = np.sort(rng.choice(S - maxlen, n, replace=False))
    out = []
    prev = 0
    for s in starts:
        s = max(int(s), prev)
        ln = int(rng.integers(1, maxlen + 1))
        if s + ln > S:
            break
        out.append((s, ln))
        prev = s + ln
    return out


def _oracle_keep(S, score, retired, pending, r_pre, B, eta, max_pages, keep_recent):
    prot_idx = O.protect_pending([p[0] for p in pending], [p[1] for p in pending], r_pre, B, eta, max_pages)
    prot = [pending[i] for i in prot_idx]
    st = O.token_states(S, retired, prot, keep_recent)
    return O.select_tokens(score, st, B), st


def _accepted_form(P, rng, allp, retired):
    """Half of the retired pages as a host list; the other half as accepted
    flags over a shuffled candidate list of a page table (with rejected
    decoys, and accepted-looking entries past n_cand that must be ignored)."""
    table = sorted(set(allp) | set(retired))
    index = {p: i for i, p in enumerate(table)}
    dev_ret, host_ret = retired[::2], retired[1::2]
    decoys = [p for p in table if p not in set(retired)][: max(1, len(dev_ret))]
    entries = [(index[p], 1) for p in dev_ret] + [(index[p], 0) for p in decoys]
    rng.shuffle(entries)
    n = len(entries)
    pad = [(index[p], 1) for p in decoys[:3]]            # beyond n_cand: ignored
    cand = torch.tensor([e[0] for e in entries + pad], dtype=torch.int32).cuda()
    flags = torch.tensor([e[1] for e in entries + pad], dtype=torch.uint8).cuda()
    n_cand = torch.tensor([n], dtype=torch.int32).cuda()
    tab = P.Pages([p[0] for p in table], [p[1] for p in table])
    return host_ret, (tab, cand, n_cand, flags, n + len(pad))


def _run(P, ctx, n_seq, n_layers, H, d, cap, n_tokens, B, seed, keep_recent=0, eta=0.125,
         max_pages=16, ties=False, nan=False, accepted=False, n_pending=40, page_div=80, maxlen=64,
         ablation=()):
    rng = np.random.default_rng(seed)
    k = torch.randint(-32768, 32767, (n_seq, n_layers, H, cap, d), dtype=torch.int16).view(torch.bfloat16).cuda()
    v = torch.randint(-32768, 32767, (n_seq, n_layers, H, cap, d), dtype=torch.int16).view(torch.bfloat16).cuda()
    pos = torch.from_numpy(np.cumsum(rng.integers(1, 3, (n_seq, cap)), axis=1).astype(np.int32)).cuda()
    stride = cap + 16
    score = np.stack([make_scores(stride, seed=seed * 10 + s, ties=ties) for s in range(n_seq)])
    if nan:
        score[:, ::97] = np.nan
        score[:, 5::101] = -0.0
    retired, pending, rpre, tables = [], [], [], []
    for s in range(n_seq):
        S = n_tokens[s]
        allp = _pages(rng, S, max(4, S // page_div), maxlen)
        rng.shuffle(allp)
        ret = sorted(allp[: len(allp) // 3])
        pen = sorted(allp[len(allp) // 3: len(allp) // 3 + n_pending])
        if s == 0 and ret and pen:
            pen = sorted(set(pen) | {ret[0]})     # a page both retired and pending
        retired.append(ret)
        tables.append(allp)
        pending.append(pen)
        r = rng.uniform(0, 1, len(pen)).astype(np.float32)
        if len(r) > 3:
            r[1] = r[2]                            # tie in R-
        rpre.append(r)
    host_retired, acc = retired, None
    if accepted:
        forms = [_accepted_form(P, rng, tables[s], retired[s]) for s in range(n_seq)]
        host_retired = [f[0] for f in forms]
        acc = [f[1] for f in forms]
    ctx.set_policy(*ablation)
    try:
        out = P.ckv_select_and_compact(
            ctx, k, v, pos, n_tokens, torch.from_numpy(score).cuda(),
            [P.Pages([p[0] for p in r], [p[1] for p in r]) for r in host_retired],
            [P.Pages([p[0] for p in r], [p[1] for p in r]) for r in pending],
            [torch.from_numpy(r).cuda() if len(r) else None for r in rpre],
            budget=B, eta=eta, max_pending_pages=max_pages, keep_recent=keep_recent, accepted=acc)
    finally:
        ctx.set_policy()
    torch.cuda.synchronize()
    # Sec. 4.4 variants on the oracle side: no protected page; no retired page
    if "no_protection" in ablation or "no_lifecycle" in ablation:
        pending = [[] for _ in pending]
        rpre = [np.zeros(0, np.float32) for _ in rpre]
    if "no_lifecycle" in ablation:
        retired = [[] for _ in retired]
    kept = out["kept"].cpu().numpy()
    nk = out["n_kept"].cpu().numpy()
    kn, vn = k.view(torch.int16).cpu().numpy(), v.view(torch.int16).cpu().numpy()
    ko, vo = out["k"].view(torch.int16).cpu().numpy(), out["v"].view(torch.int16).cpu().numpy()
    pn, po = pos.cpu().numpy(), out["pos"].cpu().numpy()
    for s in range(n_seq):
        S = n_tokens[s]
        want, _ = _oracle_keep(S, score[s, :S], retired[s], pending[s], rpre[s], B, eta, max_pages,
                               keep_recent)
        assert nk[s] == len(want), (s, nk[s], len(want))
        np.testing.assert_array_equal(kept[s, :nk[s]], want)
        assert np.all(kept[s, nk[s]:] == -1)
        np.testing.assert_array_equal(ko[s, :, :, :nk[s]], kn[s][:, :, want])
        np.testing.assert_array_equal(vo[s, :, :, :nk[s]], vn[s][:, :, want])
        np.testing.assert_array_equal(po[s, :nk[s]], pn[s, want])
    return out


def test_single_layer_d128(ckv):
    P, ctx = ckv
    _run(P, ctx, 1, 1, 8, 128, 5000, [5000], 1500, seed=1)


def test_batched_stack_d64_ties_nan(ckv):
    P, ctx = ckv
    _run(P, ctx, 3, 4, 2, 64, 3000, [3000, 2100, 777], 640, seed=2, ties=True, nan=True, keep_recent=32)


def test_budget_exceeds_cache(ckv):
    """Budget larger than the non-retired cache: every non-retired token is kept."""
    P, ctx = ckv
    _run(P, ctx, 1, 2, 2, 128, 900, [900], 1024, seed=3, eta=0.5)


def test_protection_fills_pending_budget(ckv):
    P, ctx = ckv
    _run(P, ctx, 2, 1, 1, 64, 4000, [4000, 3999], 256, seed=4, eta=1.0, max_pages=100)


def test_retired_on_device(ckv):
    """Retired pages given partly as a host list and partly as accepted
    flags over a device candidate list (the joint test's output)."""
    P, ctx = ckv
    _run(P, ctx, 2, 2, 2, 128, 6000, [6000, 4100], 1200, seed=6, keep_recent=64, accepted=True)


def test_many_sequences_with_accepted_pages(ckv):
    """20 sequences, each with its own device page table of accepted
    candidates: the call takes 20 page-table copies plus the argument blob
    that points at them, more than the copy cache's 16 entries, and none of
    the copies this call uses may be evicted before its kernels run."""
    P, ctx = ckv
    lens = [2500 + 37 * s for s in range(20)]
    _run(P, ctx, 20, 1, 1, 64, 3300, lens, 900, seed=11, keep_recent=16, accepted=True)


def test_unequal_sequences(ckv):
    """32768 and 20001 tokens in one call: the shorter sequence's last
    2048-token chunks are empty but still take part in its phases; with
    device-retired pages."""
    P, ctx = ckv
    _run(P, ctx, 2, 1, 1, 64, 32768, [32768, 20001], 8192, seed=7, keep_recent=64, accepted=True)


def test_chunk_boundary(ckv):
    """32769 tokens: one token in the last chunk; ties in the scores."""
    P, ctx = ckv
    _run(P, ctx, 1, 1, 1, 64, 32769, [32769], 8000, seed=8, keep_recent=16, ties=True)


def test_chunked_long_sequence(ckv):
    """140000 tokens, past the longest sequence the one-launch selection
    takes (64 chunks), so the chunked radix select runs."""
    P, ctx = ckv
    _run(P, ctx, 1, 1, 1, 64, 140000, [140000], 30000, seed=10, keep_recent=64, accepted=True)


def test_many_pending_pages(ckv):
    """More than 1024 short pending pages (ranked from global memory by the
    chunked path), most of them protected."""
    P, ctx = ckv
    out = _run(P, ctx, 1, 1, 1, 64, 30000, [30000], 9000, seed=9, eta=0.5, max_pages=5000,
               n_pending=1100, page_div=10, maxlen=8)
    assert int(out["n_kept"][0]) == 9000


def test_long_cache_q32b_shape(ckv):
    """131072 tokens, budget 32768 (the long-context layer shape)."""
    P, ctx = ckv
    _run(P, ctx, 1, 1, 8, 128, 131072, [131072], 32768, seed=5)


def test_host_errors(ckv):
    P, ctx = ckv
    k = torch.zeros((1, 1, 1, 64, 64), dtype=torch.bfloat16, device="cuda")
    pos = torch.zeros((1, 64), dtype=torch.int32, device="cuda")
    sc = torch.zeros((1, 64), device="cuda")
    E = P.Pages([], [])
    with pytest.raises(P.CKVError) as e:
        P.ckv_select_and_compact(ctx, k, k.clone(), pos, [64], sc, [E], [E], [None], budget=16,
                                 eta=0.5, keep_recent=9)
    assert e.value.code == -3
    with pytest.raises(P.CKVError) as e:        # output aliases the input
        P.ckv_select_and_compact(ctx, k, k.clone(), pos, [64], sc, [E], [E], [None], budget=16,
                                 k_out=k[:, :, :, :16], v_out=k[:, :, :, 16:32],
                                 pos_out=pos[:, :16].clone())
    assert e.value.code == -1
    with pytest.raises(P.CKVError) as e:        # page outside the cache
        P.ckv_select_and_compact(ctx, k, k.clone(), pos, [64], sc, [P.Pages([60], [8])], [E], [None],
                                 budget=16)
    assert e.value.code == -2


@pytest.mark.parametrize("ablation", [("no_protection",), ("no_lifecycle",)])
def test_ablation_variants(ckv, ablation):
    """Sec. 4.4: without transition protection no pending page is protected;
    without the lifecycle mechanism retired and accepted pages are kept
    eligible too (only the budget and keep_recent decide)."""
    P, ctx = ckv
    _run(P, ctx, 2, 2, 2, 128, 6000, [6000, 4100], 1200, seed=16, keep_recent=64, accepted=True,
         eta=0.5, ablation=ablation)


@pytest.mark.parametrize("mode", ["max", "mean"])
def test_pool_scores(ckv, mode):
    """The pooled base score (reading R12): max pooling bit-exact, mean
    pooling to float32 rounding; ragged sequences, ties, NaN, kernel 1."""
    P, ctx = ckv
    rng = np.random.default_rng(9)
    n_seq, stride = 3, 5000
    sc = rng.standard_normal((n_seq, stride)).astype(np.float32)
    sc[0, 100:110] = np.nan
    sc[1, ::50] = 7.0
    nt = [5000, 4321, 1]
    for k in (1, 7, 63):
        out = P.ckv_pool_scores(ctx, torch.from_numpy(sc).cuda(), nt, k, mode)
        torch.cuda.synchronize()
        out = out.cpu().numpy()
        for s in range(n_seq):
            want = O.pool_scores(sc[s, :nt[s]], k, mode)
            if mode == "max":
                np.testing.assert_array_equal(out[s, :nt[s]], want.astype(np.float32))
            else:
                np.testing.assert_allclose(out[s, :nt[s]], want, rtol=1e-5, atol=1e-5)
            assert np.all(out[s, nt[s]:] == 0)
    with pytest.raises(P.CKVError):
        P.ckv_pool_scores(ctx, torch.from_numpy(sc).cuda(), nt, 4, mode)     # even kernel
