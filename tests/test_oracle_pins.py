"""Pins of the fp64 oracle against facts the paper and the mathematics fix.

None of these compare the oracle with itself: each expected value comes from a
hand derivation, a textbook identity, a library routine, or the brute-force
definition of the deletion effect (Sec. 3.2, Eq. (6)-(7)).
"""
import math

import numpy as np
import pytest
from scipy.special import logsumexp, softmax

import oracle as O


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------------------
# deletion effect (Sec. 3.2, Eq. (6)-(7))
# ---------------------------------------------------------------------------
def test_worked_two_token_example():
    """Hand example: logits (0, ln 3) so a = (1/4, 3/4), v1 = (1,0), v2 = (0,1).

    o = (1/4, 3/4).  Deleting token 2 leaves o' = v1, so
    ||o - o'|| / ||o|| = 0.75*sqrt(2) / sqrt(0.625) = 3/sqrt(5).
    Deleting token 1 leaves o' = v2: 0.25*sqrt(2)/sqrt(0.625) = 1/sqrt(5).
    """
    K = np.array([[[0.0, 0.0], [math.log(3.0), 0.0]]])      # [Hkv=1, S=2, d=2]
    V = np.array([[[1.0, 0.0], [0.0, 1.0]]])
    Q = np.array([[[1.0, 0.0]]])                              # [Hq=1, W=1, d]
    pos, qpos = np.array([0, 1]), np.array([1])
    for method in ("bruteforce", "closed"):
        R, Rh = O.page_effects(K, V, pos, Q, qpos, [(1, 1), (0, 1)], scale=1.0,
                               method=method)
        assert R[0] == pytest.approx(3 / math.sqrt(5), rel=1e-14)
        assert R[1] == pytest.approx(1 / math.sqrt(5), rel=1e-14)
        assert np.array_equal(R, Rh[:, 0])


def _random_case(seed, Hkv=2, group=2, S=40, W=5, d=8, gapped=True):
    r = _rng(seed)
    K = r.standard_normal((Hkv, S, d)) * 1.5
    V = r.standard_normal((Hkv, S, d))
    Q = r.standard_normal((Hkv * group, W, d))
    if gapped:
        pos = np.cumsum(r.integers(1, 4, S)) - 1
    else:
        pos = np.arange(S)
    # window rows sit inside the cache tail, so causality cuts some pages
    qpos = np.sort(r.choice(pos[S // 2:], W, replace=False))
    starts = np.sort(r.choice(S - 3, 7, replace=False))
    pages = []
    for i, st in enumerate(starts):
        nxt = starts[i + 1] if i + 1 < len(starts) else S
        pages.append((int(st), int(min(r.integers(1, 6), nxt - st))))
    return K, V, Q, pos, qpos, pages


@pytest.mark.parametrize("seed", range(6))
def test_closed_form_matches_bruteforce(seed):
    K, V, Q, pos, qpos, pages = _random_case(seed)
    Rb, Rhb = O.page_effects(K, V, pos, Q, qpos, pages, method="bruteforce")
    Rc, Rhc = O.page_effects(K, V, pos, Q, qpos, pages, method="closed")
    fin = np.isfinite(Rhb)
    assert np.array_equal(fin, np.isfinite(Rhc))
    np.testing.assert_allclose(Rhc[fin], Rhb[fin], rtol=1e-10, atol=1e-300)
    np.testing.assert_allclose(Rc[np.isfinite(Rb)], Rb[np.isfinite(Rb)], rtol=1e-10)


def test_unattended_page_changes_nothing():
    """A page no window row can see (every p_i > every window position)."""
    K, V, Q, pos, _, _ = _random_case(3, gapped=False)
    S = K.shape[1]
    qpos = pos[[20, 25, 28, 30, 31]]
    late = int(np.searchsorted(pos, qpos.max(), side="right"))
    assert late < S - 2
    page = (late, S - late)
    for method in ("bruteforce", "closed"):
        R, Rh = O.page_effects(K, V, pos, Q, qpos, [page], method=method)
        assert R[0] == 0.0 and np.all(Rh == 0.0)
    # the re-run output is bit-identical to the original output
    vis = O.visibility(pos, qpos)
    s = O.head_logits(Q[0], K[0], 1 / math.sqrt(K.shape[2]))
    _, o = O.attend(s, vis, V[0])
    _, o2 = O.attend(s, vis & ~O.page_mask(S, *page)[None, :], V[0])
    assert np.array_equal(o, o2)


def test_uniform_attention_mean_identity():
    """Q = 0: equal logits, o = mean(v); deleting E gives
    ratio = (|E|/n) * ||mean(v_E) - mean(v_rest)|| / ||mean(v_all)||."""
    r = _rng(7)
    S, d = 30, 6
    K = r.standard_normal((1, S, d))
    V = r.standard_normal((1, S, d)) + 0.3
    Q = np.zeros((1, 1, d))
    pos, qpos = np.arange(S), np.array([S - 1])
    pages = [(0, 4), (10, 7), (29, 1)]
    R, _ = O.page_effects(K, V, pos, Q, qpos, pages)
    for (st, ln), got in zip(pages, R):
        m = np.zeros(S, bool)
        m[st:st + ln] = True
        vE, vR, vA = V[0][m].mean(0), V[0][~m].mean(0), V[0].mean(0)
        want = (ln / S) * np.linalg.norm(vE - vR) / np.linalg.norm(vA)
        assert got == pytest.approx(want, rel=1e-12)


def test_only_page_is_infinite():
    K, V, Q, pos, qpos, _ = _random_case(1, gapped=False)
    # window row sees tokens 0..3 only; the page covers all of them
    qpos = np.array([3])
    Q = Q[:, :1]
    R, Rh = O.page_effects(K, V, pos, Q, qpos, [(0, 4), (0, 2)])
    assert np.isinf(R[0]) and np.all(np.isinf(Rh[0]))
    assert np.isfinite(R[1])
    Rc, _ = O.page_effects(K, V, pos, Q, qpos, [(0, 4)], method="closed")
    assert np.isinf(Rc[0])


def test_value_scale_and_logit_shift_invariance():
    K, V, Q, pos, qpos, pages = _random_case(11)
    R, _ = O.page_effects(K, V, pos, Q, qpos, pages)
    R2, _ = O.page_effects(K, 3.5 * V, pos, Q, qpos, pages)
    np.testing.assert_allclose(R2, R, rtol=1e-12)
    # adding a per-row constant to every logit changes nothing
    vis = O.visibility(pos, qpos)
    s = O.head_logits(Q[0], K[0], 0.3)
    dm = O.page_mask(K.shape[1], *pages[2])
    base = O.deletion_ratio_bruteforce(s, vis, V[0], dm)
    shifted = O.deletion_ratio_bruteforce(s + np.arange(len(qpos))[:, None] * 7.0,
                                          vis, V[0], dm)
    np.testing.assert_allclose(shifted, base, rtol=1e-10)


def test_token_permutation_with_positions_carried():
    K, V, Q, pos, qpos, pages = _random_case(5)
    S = K.shape[1]
    perm = _rng(2).permutation(S)
    vis = O.visibility(pos, qpos)
    vis_p = O.visibility(pos[perm], qpos)
    for h in range(Q.shape[0]):
        g = h // 2
        s = O.head_logits(Q[h], K[g], 0.4)
        s_p = O.head_logits(Q[h], K[g][perm], 0.4)
        for st, ln in pages:
            dm = O.page_mask(S, st, ln)
            a = O.deletion_ratio_bruteforce(s, vis, V[g], dm)
            b = O.deletion_ratio_bruteforce(s_p, vis_p, V[g][perm], dm[perm])
            np.testing.assert_allclose(b, a, rtol=1e-10)


def test_gqa_equals_mha_with_replicated_kv():
    K, V, Q, pos, qpos, pages = _random_case(9, Hkv=2, group=3)
    R, Rh = O.page_effects(K, V, pos, Q, qpos, pages)
    Kr, Vr = np.repeat(K, 3, axis=0), np.repeat(V, 3, axis=0)
    R2, Rh2 = O.page_effects(Kr, Vr, pos, Q, qpos, pages)
    np.testing.assert_allclose(Rh2, Rh, rtol=1e-13)
    # a transposed GQA mapping (h % Hkv) would differ
    Kx = np.concatenate([K[[0]], K[[1]], K[[0]], K[[1]], K[[0]], K[[1]]])
    Vx = np.concatenate([V[[0]], V[[1]], V[[0]], V[[1]], V[[0]], V[[1]]])
    R3, _ = O.page_effects(Kx, Vx, pos, Q, qpos, pages)
    assert not np.allclose(R3, R)


def test_window_outputs_against_library_softmax():
    K, V, Q, pos, qpos, _ = _random_case(4)
    Ow, lse, nvis = O.window_outputs(K, V, pos, Q, qpos)
    d = K.shape[2]
    for h in range(Q.shape[0]):
        for p in range(len(qpos)):
            vis = pos <= qpos[p]
            s = (Q[h, p] @ K[h // 2][vis].T) / math.sqrt(d)
            assert lse[h, p] == pytest.approx(logsumexp(s), rel=1e-13)
            np.testing.assert_allclose(Ow[h, p], softmax(s) @ V[h // 2][vis], rtol=1e-12)
            assert nvis[p] == vis.sum()


def test_token_mass_uniform_attention():
    """Q = 0: a_{p,i} = 1/n_vis(p) on visible tokens, so the mass of token i is
    sum over rows that see i of 1/n_vis(p)."""
    S, d, W = 20, 4, 3
    K = _rng(1).standard_normal((1, S, d))
    V = _rng(2).standard_normal((1, S, d))
    Q = np.zeros((2, W, d))
    pos, qpos = np.arange(S), np.array([5, 12, 30])
    m = O.token_mass(K, V, pos, Q, qpos)
    want = np.zeros(S)
    for q in qpos:
        n = (pos <= q).sum()
        want[pos <= q] += 1.0 / n
    np.testing.assert_allclose(m, want, rtol=1e-13)


# ---------------------------------------------------------------------------
# classification (Sec. 3.2, Eq. (8)-(10))
# ---------------------------------------------------------------------------
def test_percentiles_hand_values():
    np.testing.assert_array_equal(O.percentile_ranks([0.3, 0.1, 0.5, 0.2, 0.4]),
                                  [0.5, 0.0, 1.0, 0.25, 0.75])
    np.testing.assert_array_equal(O.percentile_ranks([0.1, 0.1, 0.2]), [0.0, 0.0, 1.0])
    np.testing.assert_array_equal(O.percentile_ranks([7.0]), [0.5])
    assert O.percentile_ranks([]).size == 0


def test_lifecycle_hand_table():
    """Five pages A..E chosen by hand so each state of Eq. (10) appears once,
    with R and P landing exactly on tau and rho for B (pre) and D (pre).

    page  R-     P-    H- L-   R+     P+    H+ L+   state
    A     0.9    1.0   1  0    0.05   0.75  1  0    still active
    B     0.05   0.75  1  0    0.01   0.25  0  1    completion candidate
    C     0.001  0.0   0  1    0.002  0.0   0  1    dormant
    D     0.01   0.25  0  1    0.5    1.0   1  0    newly active
    E     0.03   0.5   0  0    0.04   0.5   0  0    uncertain
    """
    Rm = [0.9, 0.05, 0.001, 0.01, 0.03]
    Rp = [0.05, 0.01, 0.002, 0.5, 0.04]
    lam, Pm, Pp, cand = O.classify(Rm, Rp, starts=[0, 16, 32, 48, 64])
    np.testing.assert_array_equal(Pm, [1.0, 0.75, 0.0, 0.25, 0.5])
    np.testing.assert_array_equal(Pp, [0.75, 0.25, 0.0, 1.0, 0.5])
    np.testing.assert_array_equal(lam, [O.STILL_ACTIVE, O.CANDIDATE, O.DORMANT,
                                        O.NEWLY_ACTIVE, O.UNCERTAIN])
    np.testing.assert_array_equal(cand, [1])
    # just past a threshold flips the decision
    lam2, *_ = O.classify([0.9, 0.0499999, 0.001, 0.0100001, 0.03], Rp,
                          starts=[0, 16, 32, 48, 64])
    np.testing.assert_array_equal(lam2, [O.STILL_ACTIVE, O.UNCERTAIN, O.DORMANT,
                                         O.UNCERTAIN, O.UNCERTAIN])


def test_ablation_without_precommit_state():
    """Sec. 4.4: candidates from L+ alone.  In the hand table above, B (H-, L+)
    and C (L-, L+, dormant in the full method) become candidates, ordered by
    R+ ascending: C (0.002) before B (0.01); the other states are unchanged."""
    Rm = [0.9, 0.05, 0.001, 0.01, 0.03]
    Rp = [0.05, 0.01, 0.002, 0.5, 0.04]
    lam, _, _, cand = O.classify(Rm, Rp, starts=[0, 16, 32, 48, 64], ablation=("no_precommit",))
    np.testing.assert_array_equal(lam, [O.STILL_ACTIVE, O.CANDIDATE, O.CANDIDATE,
                                        O.NEWLY_ACTIVE, O.UNCERTAIN])
    np.testing.assert_array_equal(cand, [2, 1])


def test_ablation_without_percentile():
    """Sec. 4.4: every page has R- >= tau_use and R+ <= tau_dead.  With the
    percentile calibration only the top quartile is high before (pages 3, 4)
    and the bottom quartile low after (pages 0, 1), so no page is a
    candidate; with the absolute thresholds alone all five are, ordered by R+."""
    Rm = [0.2, 0.3, 0.4, 0.5, 0.6]
    Rp = [0.001, 0.002, 0.003, 0.004, 0.005]
    st = [0, 16, 32, 48, 64]
    lam, _, _, cand = O.classify(Rm, Rp, st)
    assert cand.size == 0 and not np.any(lam == O.CANDIDATE)
    lam2, _, _, cand2 = O.classify(Rm, Rp, st, ablation=("no_percentile",))
    assert np.all(lam2 == O.CANDIDATE)
    np.testing.assert_array_equal(cand2, [0, 1, 2, 3, 4])


def test_ablation_without_lifecycle_has_no_candidate():
    lam, _, _, cand = O.classify([0.9, 0.05], [0.001, 0.002], starts=[0, 16], ablation=("no_lifecycle",))
    assert cand.size == 0


def test_high_needs_both_absolute_and_percentile():
    """A page ranked first among tiny effects is not high (Sec. 3.2)."""
    H, L = O.high_low(np.array([0.02, 0.001]), np.array([1.0, 0.0]),
                      0.05, 0.01, 0.75, 0.25)
    assert not H[0] and not L[0] and L[1]


def test_candidate_order():
    """R+ ascending, then R- descending, then start ascending."""
    Rm = [0.9, 0.8, 0.9, 0.7, 0.001, 0.002, 0.003, 0.004, 0.0, 0.0, 0.0005, 0.0006, 0.0007]
    Rp = [0.001, 0.001, 0.001, 0.0005, 0.2, 0.3, 0.4, 0.5, 0.6, 0.7, 0.8, 0.9, 1.0]
    starts = [40, 10, 20, 30, 0, 50, 60, 70, 80, 90, 100, 110, 120]
    lam, _, _, cand = O.classify(Rm, Rp, starts)
    assert set(cand.tolist()) == {0, 1, 2, 3}
    np.testing.assert_array_equal(cand, [3, 2, 0, 1])
    _, _, _, capped = O.classify(Rm, Rp, starts, max_cand=2)
    np.testing.assert_array_equal(capped, [3, 2])


def _lifecycle_attention_case():
    """Five 4-token pages with hand-set keys (d = 4, scale 1):
    X = (2,-2,0,0): pre logit +6, post -6   -> high-to-low
    Y = (-2,-2,0,0): pre -6, post -6        -> low-to-low
    Z = (2,2,0,0): +6, +6; Wn = (-2,2,0,0): -6, +6; F = 0: 0, 0.
    Pre window rows query (3,0,0,0); post rows query (0,3,0,0).
    """
    keys = [(2, -2), (-2, -2), (2, 2), (-2, 2), (0, 0)]
    S, d = 20, 4
    K = np.zeros((1, S, d))
    for j, (a, b) in enumerate(keys):
        K[0, 4 * j:4 * j + 4, 0] = a
        K[0, 4 * j:4 * j + 4, 1] = b
    V = _rng(3).standard_normal((1, S, d))
    Qm = np.zeros((1, 2, d)); Qm[0, :, 0] = 3.0
    Qp = np.zeros((1, 2, d)); Qp[0, :, 1] = 3.0
    pos, qpos = np.arange(S), np.array([100, 101])
    pages = [(4 * j, 4) for j in range(5)]
    return K, V, Qm, Qp, pos, qpos, pages


def test_hand_built_candidate_and_dormant():
    K, V, Qm, Qp, pos, qpos, pages = _lifecycle_attention_case()
    Rm, _ = O.page_effects(K, V, pos, Qm, qpos, pages, scale=1.0)
    Rp, _ = O.page_effects(K, V, pos, Qp, qpos, pages, scale=1.0)
    lam, _, _, cand = O.classify(Rm, Rp, [p[0] for p in pages])
    assert lam[0] == O.CANDIDATE
    assert lam[1] == O.DORMANT
    assert lam[2] == O.STILL_ACTIVE
    assert lam[3] == O.NEWLY_ACTIVE
    np.testing.assert_array_equal(cand, [0])


# ---------------------------------------------------------------------------
# joint test (Sec. 3.3, Eq. (11), Algorithm 1)
# ---------------------------------------------------------------------------
def test_union_of_one_page_is_its_own_effect():
    K, V, Q, pos, qpos, pages = _random_case(8)
    R, _ = O.page_effects(K, V, pos, Q, qpos, pages)
    for j in range(len(pages)):
        assert O.union_effect(K, V, pos, Q, qpos, pages, [j]) == pytest.approx(R[j], rel=1e-12)


def _two_small_pages():
    """Uniform attention over n = 400 tokens with v = (1, 0) except two 4-token
    pages with v = (1, 0.8).  By the mean identity each page alone moves the
    output by ~0.0079 and both together by ~0.0157, around tau_joint = 0.01."""
    S = 400
    K = np.zeros((1, S, 2))
    V = np.zeros((1, S, 2)); V[0, :, 0] = 1.0
    V[0, 100:104, 1] = 0.8
    V[0, 200:204, 1] = 0.8
    Q = np.zeros((1, 3, 2))
    pos, qpos = np.arange(S), np.array([S, S + 1, S + 2])
    pages = [(100, 4), (200, 4), (300, 4)]
    return K, V, Q, pos, qpos, pages


def _mean_identity(V, mask):
    n = V.shape[0]
    vE, vR, vA = V[mask].mean(0), V[~mask].mean(0), V.mean(0)
    return (mask.sum() / n) * np.linalg.norm(vE - vR) / np.linalg.norm(vA)


def test_joint_rejects_accumulated_effect():
    K, V, Q, pos, qpos, pages = _two_small_pages()
    S = K.shape[1]
    m1, m2 = O.page_mask(S, 100, 4), O.page_mask(S, 200, 4)
    r1, r12 = _mean_identity(V[0], m1), _mean_identity(V[0], m1 | m2)
    assert r1 < 0.01 < r12
    acc, uR = O.joint_test(K, V, pos, Q, qpos, pages, [0, 1, 2], tau_joint=0.01)
    np.testing.assert_array_equal(acc, [True, False, True])
    assert uR[0] == pytest.approx(r1, rel=1e-12)
    assert uR[1] == pytest.approx(r12, rel=1e-12)
    # page 2 carries v = (1,0) like the rest, A u {2} only renormalises
    assert uR[2] == pytest.approx(_mean_identity(V[0], m1 | O.page_mask(S, 300, 4)), rel=1e-12)


def test_ablation_without_joint_validation_accepts_all():
    """Sec. 4.4: without the Eq. (11) gate both small pages are retired, and
    the union effects follow the mean identity for {0}, {0,1}, {0,1,2}."""
    K, V, Q, pos, qpos, pages = _two_small_pages()
    S = K.shape[1]
    m = [O.page_mask(S, st, ln) for st, ln in pages]
    acc, uR = O.joint_test(K, V, pos, Q, qpos, pages, [0, 1, 2], tau_joint=0.01, gate=False)
    np.testing.assert_array_equal(acc, [True, True, True])
    assert uR[1] == pytest.approx(_mean_identity(V[0], m[0] | m[1]), rel=1e-12)
    assert uR[2] == pytest.approx(_mean_identity(V[0], m[0] | m[1] | m[2]), rel=1e-12)
    assert uR[1] > 0.01


def test_first_candidate_always_accepted():
    """tau_joint >= tau_dead and the first candidate is L+, so
    R+({E}) = R+(E) <= tau_dead <= tau_joint."""
    K, V, Qm, Qp, pos, qpos, pages = _lifecycle_attention_case()
    Rm, _ = O.page_effects(K, V, pos, Qm, qpos, pages, scale=1.0)
    Rp, _ = O.page_effects(K, V, pos, Qp, qpos, pages, scale=1.0)
    _, _, _, cand = O.classify(Rm, Rp, [p[0] for p in pages])
    acc, uR = O.joint_test(K, V, pos, Qp, qpos, pages, cand, tau_joint=0.01, scale=1.0)
    assert acc[0] and uR[0] == pytest.approx(Rp[cand[0]], rel=1e-12)


def test_joint_closed_form_equals_bruteforce():
    K, V, Q, pos, qpos, pages = _random_case(12)
    cand = [4, 0, 2, 6, 1]
    a1, u1 = O.joint_test(K, V, pos, Q, qpos, pages, cand, tau_joint=0.2)
    a2, u2 = O.joint_test(K, V, pos, Q, qpos, pages, cand, tau_joint=0.2, method="closed")
    np.testing.assert_array_equal(a1, a2)
    np.testing.assert_allclose(u2, u1, rtol=1e-10)
    rep = O.joint_replay(K, V, pos, Q, qpos, pages, cand, a1)
    np.testing.assert_allclose(rep, u1, rtol=1e-14)


# ---------------------------------------------------------------------------
# checkpoint (Sec. 3.3, Eq. (12)-(13); Sec. 3.1, Eq. (4))
# ---------------------------------------------------------------------------
def test_pending_budget_floor():
    assert O.pending_budget(1024, 0.125) == 128
    assert O.pending_budget(7, 0.5) == 3
    assert O.pending_budget(8192, 0.125) == 1024
    assert O.pending_budget(10, 0.0) == 0


def test_protect_pending_prefix_rule():
    """B = 64, eta = 1/8 -> B_N = 8.  Order by R- desc, start asc:
    p1 (0.9, 4 tok), p2 (0.7, start 8, 2 tok), p3 (0.7, start 10, 4 tok), p0, p4.
    p1 + p2 = 6 tokens; p3 would make 10 > 8 -> stop (p4 is not tried)."""
    starts = [0, 4, 8, 10, 14]
    lens = [4, 4, 2, 4, 1]
    Rm = [0.5, 0.9, 0.7, 0.7, 0.1]
    np.testing.assert_array_equal(O.protect_pending(starts, lens, Rm, 64, 0.125), [1, 2])
    np.testing.assert_array_equal(O.protect_pending(starts, lens, Rm, 64, 0.125, max_pages=1), [1])
    np.testing.assert_array_equal(O.protect_pending(starts, lens, Rm, 200, 0.125), [1, 2, 3, 0, 4])
    assert O.protect_pending(starts, lens, Rm, 16, 0.125).size == 0


def test_token_states_precedence():
    st = O.token_states(20, retired_pages=[(2, 3), (10, 2)], protected_pages=[(3, 4)],
                        keep_recent=3)
    want = np.zeros(20, np.uint8)
    want[[3, 4, 5, 6, 17, 18, 19]] = O.PROTECTED
    want[[2, 3, 4, 10, 11]] = O.RETIRED
    np.testing.assert_array_equal(st, want)


@pytest.mark.parametrize("seed", range(4))
def test_select_matches_lexsort(seed):
    r = _rng(seed)
    S, B = 300, 90
    score = np.round(r.standard_normal(S) * 3).astype(np.float32)   # many ties
    state = r.choice([O.FREE, O.FREE, O.FREE, O.PROTECTED, O.RETIRED], S).astype(np.uint8)
    state[:] = np.where(np.arange(S) % 17 == 0, O.PROTECTED, state)
    nprot = int((state == O.PROTECTED).sum())
    keep = O.select_tokens(score, state, B + nprot)
    free = np.flatnonzero(state == O.FREE)
    order = np.lexsort((free, -score[free].astype(np.float64)))
    want = np.sort(np.concatenate([np.flatnonzero(state == O.PROTECTED), free[order[:B]]]))
    np.testing.assert_array_equal(keep, want)
    assert len(keep) <= B + nprot
    assert np.all(np.diff(keep) > 0)
    assert not np.any(state[keep] == O.RETIRED)


def test_select_edge_cases():
    state = np.zeros(6, np.uint8)
    # fewer free tokens than the budget: keep every non-retired token
    state[2] = O.RETIRED
    np.testing.assert_array_equal(O.select_tokens(np.zeros(6, np.float32), state, 100),
                                  [0, 1, 3, 4, 5])
    # -0.0 ties +0.0 and NaN ties -inf (the lower index wins a tie)
    score = np.array([np.nan, -0.0, 0.0, -np.inf, 1.0, -0.0], np.float32)
    np.testing.assert_array_equal(O.select_tokens(score, np.zeros(6, np.uint8), 3), [1, 2, 4])
    np.testing.assert_array_equal(O.select_tokens(score, np.zeros(6, np.uint8), 5), [0, 1, 2, 4, 5])
    # protected tokens beyond the budget are an error
    with pytest.raises(ValueError):
        O.select_tokens(np.zeros(4, np.float32), np.full(4, O.PROTECTED, np.uint8), 3)
    assert O.select_tokens(np.zeros(0, np.float32), np.zeros(0, np.uint8), 4).size == 0


def test_compaction_is_one_index_set():
    r = _rng(0)
    K = r.integers(0, 2**16, (3, 2, 10, 4)).astype(np.uint16)
    V = r.integers(0, 2**16, (3, 2, 10, 4)).astype(np.uint16)
    pos = np.cumsum(r.integers(1, 5, 10)).astype(np.int32)
    keep = np.array([0, 3, 4, 9])
    Kc, Vc, pc = O.compact(K, V, pos, keep)
    for j, i in enumerate(keep):
        assert np.array_equal(Kc[:, :, j], K[:, :, i])
        assert np.array_equal(Vc[:, :, j], V[:, :, i])
        assert pc[j] == pos[i]


# ---------------------------------------------------------------- pooled base score (R12)
def test_pool_max_equals_library_filter():
    from scipy.ndimage import maximum_filter1d
    x = np.random.default_rng(5).standard_normal(300)
    for k in (1, 3, 7, 31):
        np.testing.assert_array_equal(O.pool_scores(x, k, "max"), maximum_filter1d(x, k, mode="nearest"))


def test_pool_mean_hand_example():
    np.testing.assert_allclose(O.pool_scores([1, 2, 3, 4, 5], 3, "mean"), [1.5, 2, 3, 4, 4.5])
    np.testing.assert_allclose(O.pool_scores([1, 2, 3, 4, 5], 5, "mean"), [2, 2.5, 3, 3.5, 4])


def test_pool_identity_and_nan():
    x = np.array([0.3, -1.0, 2.0, np.nan, 0.5])
    np.testing.assert_array_equal(O.pool_scores(x[:3], 1, "max"), x[:3])
    np.testing.assert_array_equal(O.pool_scores(x, 3, "max"), [0.3, 2.0, 2.0, 2.0, 0.5])
    assert np.isnan(O.pool_scores(x, 3, "mean")[2]) and O.pool_scores(x, 3, "mean")[0] == (0.3 - 1.0) / 2


def test_bf16_bits_decode_hand_patterns():
    """The oracle's bf16 decoder on hand-written bit patterns (sign,
    exponent, mantissa read off by hand): ones, a fraction, zeros of both
    signs, infinities, NaN, the largest finite value and the smallest
    subnormal."""
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x3C00, 0x0000, 0x8000, 0x7F80, 0xFF80, 0x7F7F, 0x0001,
                     0x4120, 0xC2F7], dtype=np.uint16)
    want = [1.0, -1.0, 3.140625, 2.0 ** -7, 0.0, -0.0, np.inf, -np.inf, (2 - 2.0 ** -7) * 2.0 ** 127,
            2.0 ** -133, 10.0, -123.5]
    got = O.bf16_bits_to_f64(bits)
    assert got.dtype == np.float64
    np.testing.assert_array_equal(got, want)
    assert np.signbit(got[5]) and not np.signbit(got[4])
    assert np.isnan(O.bf16_bits_to_f64(np.array([0x7FC0], np.uint16)))[0]
    # as_f64 takes the same path for uint16 input and leaves real arrays as they are
    np.testing.assert_array_equal(O.as_f64(bits), got)
    np.testing.assert_array_equal(O.as_f64(np.array([0.5, -2.0], np.float32)), [0.5, -2.0])
