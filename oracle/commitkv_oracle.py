"""fp64 CPU oracle for the CommitKV hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  The HIP library
never calls it, and it shares no code, constants or helpers with the HIP path.

Every function restates the paper (CommitKV, "Lifecycle-Aware KV Cache
Compression via Commit Transitions for Multi-Turn Agents") in plain NumPy
float64, in the order and notation of Sec. 3:

* Sec. 3.1, Eq. (4): compression applies one index set I to K, V and positions.
* Sec. 3.1, Eq. (5): paired query windows Q^- and Q^+.
* Sec. 3.2, Eq. (6): output of a head after deleting page E and renormalising.
* Sec. 3.2, Eq. (7): window deletion effect R_h (max over window rows) and
  R (max over heads).
* Sec. 3.2, Eq. (8): pre/post-commit effects; percentile ranks over E_c.
* Sec. 3.2, Eq. (9)-(10): high/low indicators and lifecycle states.
* Sec. 3.3, Eq. (11) and Algorithm 1: greedy joint retirement test.
* Sec. 3.3, Eq. (12)-(13): pending-page protection and the retained set.
* Sec. 4.4: the ablation variants (``ABLATIONS``) switch single components off.

The deletion effect is defined by brute force (``page_effects_bruteforce``):
attention is run again with the page masked out.  ``page_effects_closed_form``
evaluates Eq. (6) instead; both are kept so that one pins the other.

Readings taken where the paper is silent:

* R1  softmax scale 1/sqrt(d); inputs are post-RoPE keys and queries.
* R2  grouped-query attention: query head h reads KV head h // (Hq/Hkv);
      the max in Eq. (7) runs over query heads.
* R3  visibility is by absolute position, pos[i] <= qpos[p], including the
      window's own resident tokens.
* R4  a row that sees no token of E contributes 0; a row whose only visible
      tokens are in E gives +inf; ||o|| = 0 gives 0 if o' == o else +inf.
* R5  percentile P(E) = #{E' != E : R(E') < R(E)} / (n - 1); ties share the
      lower rank; n == 1 gives 0.5.
* R6  candidates are ordered by (R+ ascending, R- descending, start
      ascending); the joint test starts from an empty set at every commit
      (Algorithm 1) and deletes the union at once.
* R7  pending protection takes pages by (R- descending, start ascending)
      while fewer than max_pages are taken and the token count stays within
      B_N = floor(eta * B); it stops at the first page that does not fit.
* R8  token states: retired > protected > free; the last ``keep_recent``
      resident tokens count as protected.
* R9  the budget is filled with the free tokens of highest score, ties to the
      lower index; NaN scores count as -inf and -0.0 as +0.0; the retained
      index set is returned in ascending order.
* R10 the base score used to fill the budget is the SnapKV-style window mass
      max_h sum_{p in Q+} a_{h,p,i} (``token_mass``); the selection accepts
      any float32 score.
* R12 the pooled variant of the base score (``pool_scores``) smooths the
      aggregated score over the odd window [t - k//2, t + k//2] clipped to
      the cache: max pooling ignores NaN entries (NaN only if all are), mean
      pooling divides the window's sum by the number of tokens in it.
"""
from __future__ import annotations

import math

import numpy as np

# lifecycle state codes (Sec. 3.2, Eq. (10))
UNCERTAIN, CANDIDATE, DORMANT, NEWLY_ACTIVE, STILL_ACTIVE = 0, 1, 2, 3, 4
# token states at a compression checkpoint (Sec. 3.3, Eq. (13))
FREE, PROTECTED, RETIRED = 0, 1, 2

# Sec. 4.1 (implementation details)
PAPER_THRESHOLDS = dict(tau_use=0.05, tau_dead=0.01, rho_use=0.75,
                        rho_dead=0.25, tau_joint=0.01)

# Sec. 4.4 ablation variants, each switching one component of the method off:
#   no_precommit  retirement candidates from L+ alone instead of (H-, L+)
#   no_percentile high/low from the absolute thresholds only (no rho test)
#   no_joint      every candidate retired without the Eq. (11) gate
#   no_protection no pending page protected (N_j empty)
#   no_lifecycle  no lifecycle operation at all: nothing retired or protected
ABLATIONS = ("no_precommit", "no_percentile", "no_joint", "no_protection", "no_lifecycle")


# ----------------------------------------------------------------------------
# inputs
# ----------------------------------------------------------------------------
def bf16_bits_to_f64(bits):
    """Exact value of bfloat16 bit patterns (uint16) as float64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def as_f64(x):
    """Accept bf16 bit patterns (uint16) or real arrays; return float64."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f64(x)
    return x.astype(np.float64)


# ----------------------------------------------------------------------------
# attention of one head over the resident cache (Sec. 3.2, notation of Eq. (6))
# ----------------------------------------------------------------------------
def head_logits(q, k, scale):
    """s[p, i] = scale * q_p . k_i  (q: [W, d], k: [S, d])."""
    return scale * (q @ k.T)


def visibility(pos, qpos):
    """vis[p, i] = (p_i <= p): token i is visible from window position p."""
    return np.asarray(pos)[None, :] <= np.asarray(qpos)[:, None]


def attend(s, vis, v):
    """Softmax over the visible tokens of each row, then o_p = sum_i a_pi v_i.

    Returns (a [W, S], o [W, d]); a row with no visible token has a = 0, o = 0.
    """
    masked = np.where(vis, s, -np.inf)
    m = masked.max(axis=1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.where(vis, np.exp(masked - m), 0.0)
    z = e.sum(axis=1, keepdims=True)
    a = np.divide(e, z, out=np.zeros_like(e), where=z > 0)
    return a, a @ v


def _relative_change(o, o_del, undefined_rows):
    """||o - o'|| / ||o|| per row, with the conventions of reading R4."""
    diff = np.linalg.norm(o - o_del, axis=1)
    norm = np.linalg.norm(o, axis=1)
    out = np.empty(o.shape[0])
    for p in range(o.shape[0]):
        if undefined_rows[p]:
            out[p] = np.inf
        elif norm[p] > 0:
            out[p] = diff[p] / norm[p]
        else:
            out[p] = 0.0 if diff[p] == 0 else np.inf
    return out


def deletion_ratio_bruteforce(s, vis, v, delete):
    """Per-row ||o_p - o_p^{\\E}|| / ||o_p|| with E deleted by re-running attention.

    ``delete`` is a boolean mask over tokens (the page, or a union of pages).
    This is the definition the closed form of Eq. (6) must reproduce.
    """
    _, o = attend(s, vis, v)
    vis_del = vis & ~delete[None, :]
    _, o_del = attend(s, vis_del, v)
    touched = (vis & delete[None, :]).any(axis=1)
    emptied = touched & ~vis_del.any(axis=1)
    return _relative_change(o, o_del, emptied)


def deletion_ratio_closed_form(a, o, v, delete, vis):
    """Per-row ratio from Eq. (6): o^{\\E} = (o - sum_E a v) / (1 - sum_E a).

    Then o - o^{\\E} = (u - A o) / (1 - A) with A = sum_{i in E, visible} a_pi
    and u = sum_{i in E, visible} a_pi v_i.
    """
    sel = vis & delete[None, :]
    a_e = np.where(sel, a, 0.0)
    A = a_e.sum(axis=1)
    u = a_e @ v
    touched = sel.any(axis=1)
    emptied = touched & ~(vis & ~delete[None, :]).any(axis=1)
    norm = np.linalg.norm(o, axis=1)
    num = np.linalg.norm(u - A[:, None] * o, axis=1)
    ratio = np.zeros(o.shape[0])
    for p in range(o.shape[0]):
        if not touched[p]:
            ratio[p] = 0.0
        elif emptied[p]:
            ratio[p] = np.inf
        elif norm[p] > 0:
            ratio[p] = num[p] / ((1.0 - A[p]) * norm[p])
        else:
            ratio[p] = 0.0 if num[p] == 0 else np.inf
    return ratio


# ----------------------------------------------------------------------------
# window deletion effects of pages (Sec. 3.2, Eq. (7)-(8))
# ----------------------------------------------------------------------------
def _prep(K, V, pos, Q, qpos, scale):
    K, V, Q = as_f64(K), as_f64(V), as_f64(Q)
    Hkv, S, d = K.shape
    Hq = Q.shape[0]
    if Hq % Hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    vis = visibility(np.asarray(pos)[:S], qpos)
    return K, V, Q, Hq // Hkv, scale, vis


def page_mask(S, start, length):
    m = np.zeros(S, dtype=bool)
    m[start:start + length] = True
    return m


def page_effects(K, V, pos, Q, qpos, pages, scale=None, method="bruteforce",
                 heads=None):
    """R(E; Q) for every page E = (start, len) of ``pages``.

    K, V: [Hkv, S, d]; Q: [Hq, W, d]; pos: [S] absolute positions; qpos: [W].
    Returns (R [n], R_h [n, Hq]).  ``method`` is "bruteforce" (definition) or
    "closed" (Eq. (6)).  ``heads`` restricts the query heads evaluated (the
    remaining columns of R_h are NaN and R is the max over the given heads).
    """
    K, V, Q, group, scale, vis = _prep(K, V, pos, Q, qpos, scale)
    S = K.shape[1]
    Hq = Q.shape[0]
    heads = range(Hq) if heads is None else heads
    pages = [(int(s0), int(l0)) for s0, l0 in pages]
    R_h = np.full((len(pages), Hq), np.nan)
    for h in heads:
        g = h // group
        s = head_logits(Q[h], K[g], scale)
        if method == "closed":
            a, o = attend(s, vis, V[g])
        for j, (st, ln) in enumerate(pages):
            dm = page_mask(S, st, ln)
            if method == "closed":
                r = deletion_ratio_closed_form(a, o, V[g], dm, vis)
            else:
                r = deletion_ratio_bruteforce(s, vis, V[g], dm)
            R_h[j, h] = r.max() if r.size else 0.0
    R = np.nanmax(R_h, axis=1) if len(pages) else np.zeros(0)
    return R, R_h


def window_outputs(K, V, pos, Q, qpos, scale=None):
    """Full window attention: O [Hq, W, d], LSE [Hq, W] (natural log), n_vis [W]."""
    K, V, Q, group, scale, vis = _prep(K, V, pos, Q, qpos, scale)
    Hq, W, d = Q.shape
    O = np.zeros((Hq, W, d))
    LSE = np.full((Hq, W), -np.inf)
    for h in range(Hq):
        s = head_logits(Q[h], K[h // group], scale)
        _, O[h] = attend(s, vis, V[h // group])
        masked = np.where(vis, s, -np.inf)
        m = masked.max(axis=1)
        ok = np.isfinite(m)
        LSE[h, ok] = m[ok] + np.log(np.exp(masked[ok] - m[ok, None]).sum(axis=1))
    return O, LSE, vis.sum(axis=1)


def token_mass(K, V, pos, Q, qpos, scale=None):
    """Reading R10: score_i = max_h sum_p a_{h,p,i} (0 if no row sees token i)."""
    K, V, Q, group, scale, vis = _prep(K, V, pos, Q, qpos, scale)
    S = K.shape[1]
    out = np.zeros(S)
    for h in range(Q.shape[0]):
        s = head_logits(Q[h], K[h // group], scale)
        a, _ = attend(s, vis, V[h // group])
        out = np.maximum(out, a.sum(axis=0))
    return out


# ----------------------------------------------------------------------------
# classification (Sec. 3.2, Eq. (8)-(10))
# ----------------------------------------------------------------------------
def percentile_ranks(R):
    """Reading R5: fraction of the other pages of E_c with a strictly smaller R."""
    R = np.asarray(R, dtype=np.float64)
    n = R.size
    if n == 0:
        return np.zeros(0)
    if n == 1:
        return np.array([0.5])
    less = np.array([(R < R[j]).sum() for j in range(n)], dtype=np.float64)
    return less / (n - 1)


def high_low(R, P, tau_use, tau_dead, rho_use, rho_dead, percentile=True):
    """Eq. (9): H = (R >= tau_use and P >= rho_use); L = (R <= tau_dead and P <= rho_dead).

    percentile=False is the Sec. 4.4 variant without percentile calibration:
    the absolute thresholds alone decide.
    """
    R = np.asarray(R, dtype=np.float64)
    H = R >= tau_use
    L = R <= tau_dead
    if percentile:
        H = H & (P >= rho_use)
        L = L & (P <= rho_dead)
    return H, L


def lifecycle(H_pre, L_pre, H_post, L_post, precommit=True):
    """Eq. (10): candidate (H-,L+), dormant (L-,L+), newly active (L-,H+),
    still active (H-,H+), otherwise uncertain.

    precommit=False is the Sec. 4.4 variant without the pre-commit state:
    every page with L+ is a candidate, whatever its pre-commit state.
    """
    lam = np.full(len(H_pre), UNCERTAIN, dtype=np.uint8)
    lam[L_pre & H_post] = NEWLY_ACTIVE
    lam[H_pre & H_post] = STILL_ACTIVE
    if precommit:
        lam[H_pre & L_post] = CANDIDATE
        lam[L_pre & L_post] = DORMANT
    else:
        lam[L_post] = CANDIDATE
    return lam


def classify(R_pre, R_post, starts, tau_use=0.05, tau_dead=0.01, rho_use=0.75,
             rho_dead=0.25, max_cand=None, ablation=()):
    """Pages of E_c -> (lambda, P_pre, P_post, ordered candidate indices).

    Candidate order (Sec. 3.3 and Algorithm 1): R+ ascending, then R-
    descending, then page start ascending (reading R6).  ``ablation`` names
    Sec. 4.4 variants (``ABLATIONS``); with no_lifecycle there is no candidate.
    """
    R_pre = np.asarray(R_pre, dtype=np.float64)
    R_post = np.asarray(R_post, dtype=np.float64)
    pct = "no_percentile" not in ablation
    P_pre, P_post = percentile_ranks(R_pre), percentile_ranks(R_post)
    H_pre, L_pre = high_low(R_pre, P_pre, tau_use, tau_dead, rho_use, rho_dead, pct)
    H_post, L_post = high_low(R_post, P_post, tau_use, tau_dead, rho_use, rho_dead, pct)
    lam = lifecycle(H_pre, L_pre, H_post, L_post, "no_precommit" not in ablation)
    idx = [] if "no_lifecycle" in ablation else [j for j in range(len(lam)) if lam[j] == CANDIDATE]
    idx.sort(key=lambda j: (R_post[j], -R_pre[j], int(starts[j])))
    if max_cand is not None:
        idx = idx[:max_cand]
    return lam, P_pre, P_post, np.array(idx, dtype=np.int64)


# ----------------------------------------------------------------------------
# greedy joint test (Sec. 3.3, Eq. (11), Algorithm 1)
# ----------------------------------------------------------------------------
def union_effect(K, V, pos, Q, qpos, pages, members, scale=None,
                 method="bruteforce"):
    """R+(A) with every token of the pages in ``members`` deleted at once."""
    K, V, Q, group, scale, vis = _prep(K, V, pos, Q, qpos, scale)
    S = K.shape[1]
    dm = np.zeros(S, dtype=bool)
    for j in members:
        st, ln = pages[j]
        dm |= page_mask(S, int(st), int(ln))
    best = 0.0
    for h in range(Q.shape[0]):
        g = h // group
        s = head_logits(Q[h], K[g], scale)
        if method == "closed":
            a, o = attend(s, vis, V[g])
            r = deletion_ratio_closed_form(a, o, V[g], dm, vis)
        else:
            r = deletion_ratio_bruteforce(s, vis, V[g], dm)
        if r.size:
            best = max(best, float(r.max()))
    return best


def joint_test(K, V, pos, Q, qpos, pages, cand, tau_joint=0.01, scale=None,
               method="bruteforce", gate=True):
    """Algorithm 1: A = {}; for E in order: accept iff R+(A u {E}) <= tau_joint.

    gate=False is the Sec. 4.4 variant without joint validation: every
    candidate is accepted (union_R still reports R+(A u {E})).
    Returns (accepted bool[len(cand)], union_R float64[len(cand)]).
    """
    accepted = np.zeros(len(cand), dtype=bool)
    union_R = np.zeros(len(cand))
    A = []
    for t, j in enumerate(cand):
        r = union_effect(K, V, pos, Q, qpos, pages, A + [int(j)], scale, method)
        union_R[t] = r
        if r <= tau_joint or not gate:
            A.append(int(j))
            accepted[t] = True
    return accepted, union_R


def joint_replay(K, V, pos, Q, qpos, pages, cand, decisions, scale=None,
                 method="bruteforce"):
    """Union effect of each candidate given someone else's earlier decisions.

    Used to check a decision sequence step by step: entry t is
    R+(A_t u {E_t}) where A_t holds the candidates before t marked accepted
    in ``decisions``.
    """
    out = np.zeros(len(cand))
    A = []
    for t, j in enumerate(cand):
        out[t] = union_effect(K, V, pos, Q, qpos, pages, A + [int(j)], scale,
                              method)
        if decisions[t]:
            A.append(int(j))
    return out


# ----------------------------------------------------------------------------
# checkpoint: protection, retained set, compaction (Sec. 3.3, Eq. (12)-(13), Eq. (4))
# ----------------------------------------------------------------------------
def pending_budget(B, eta):
    """Eq. (12): B_N = floor(eta * B)."""
    return int(math.floor(eta * B))


def protect_pending(starts, lens, R_pre, B, eta=0.125, max_pages=16):
    """Eq. (12) with reading R7; returns indices of the protected pending pages."""
    BN = pending_budget(B, eta)
    order = sorted(range(len(starts)), key=lambda j: (-float(R_pre[j]), int(starts[j])))
    taken, tokens = [], 0
    for j in order:
        if len(taken) >= max_pages or tokens + int(lens[j]) > BN:
            break
        taken.append(j)
        tokens += int(lens[j])
    return np.array(taken, dtype=np.int64)


def token_states(S, retired_pages, protected_pages, keep_recent=0):
    """Reading R8: retired > protected > free, one state per resident token."""
    st = np.full(S, FREE, dtype=np.uint8)
    if keep_recent > 0:
        st[max(0, S - keep_recent):] = PROTECTED
    for s0, l0 in protected_pages:
        st[s0:s0 + l0] = PROTECTED
    for s0, l0 in retired_pages:
        st[s0:s0 + l0] = RETIRED
    return st


def select_tokens(score, state, B):
    """Eq. (13): N_j subset of I_j, |I_j| <= B, retired tokens excluded.

    Protected tokens are all kept; the remaining B - |N_j| slots go to the
    free tokens of highest float32 score, ties to the lower index (reading R9).
    Returns the ascending index set I_j; raises ValueError if |N_j| > B.
    """
    score = np.asarray(score, dtype=np.float32).astype(np.float64)
    score = np.where(np.isnan(score), -np.inf, score)
    score = np.where(score == 0, 0.0, score)          # -0.0 ranks as +0.0
    state = np.asarray(state)
    prot = np.flatnonzero(state == PROTECTED)
    free = np.flatnonzero(state == FREE)
    if prot.size > B:
        raise ValueError("protected tokens exceed the budget")
    k = min(B - prot.size, free.size)
    ranked = sorted(free.tolist(), key=lambda i: (-score[i], i))
    keep = np.array(sorted(prot.tolist() + ranked[:k]), dtype=np.int64)
    return keep


def pool_scores(score, kernel, mode="max"):
    """Reading R12: pooled base score, one output per token."""
    x = np.asarray(score, dtype=np.float64)
    n, h = x.size, kernel // 2
    out = np.empty(n)
    for t in range(n):
        win = x[max(0, t - h):min(n, t + h + 1)]
        if mode == "max":
            out[t] = np.nan if np.all(np.isnan(win)) else np.nanmax(win)
        else:
            out[t] = win.sum() / win.size
    return out


def compact(K, V, pos, keep):
    """Eq. (4): K~ = K[..., I, :], V~ = V[..., I, :], p~ = p[I] (same indices).

    K, V: [..., S, d] arrays of any dtype (copied verbatim); pos: [S].
    """
    keep = np.asarray(keep, dtype=np.int64)
    return K[..., keep, :], V[..., keep, :], np.asarray(pos)[keep]
