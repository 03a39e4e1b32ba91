"""GPU parity of ckv_joint_test (Sec. 3.3, Eq. (11), Algorithm 1).

Replay rule: the GPU's candidate order and decisions are fed to the oracle;
at each step the oracle's union effect R+(A u {E}) (brute force, all union
tokens deleted at once) must match the GPU's union_R within 2e-3, and each
decision must equal (R_ref <= tau_joint) unless R_ref is within 2e-3 of tau.
"""
import numpy as np
import pytest
import torch

import oracle as O
from synth import WORKLOADS, bf16_bits, make_layer, scaled
from tests.gpu_util import LayerOnDevice, REL_TOL, assert_scores_close, dev_bf16, dev_i32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _post_measure(P, ctx, dl):
    L = dl.L
    kv = P.kv_view(dl.k, dl.v, dl.pos)
    win = P.window_view(dl.q_post, dl.qpos_post)
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    m = P.ckv_measure_page_effects(ctx, kv, win, pages, want=("R", "o", "lse"))
    return kv, win, pages, m


def _check_replay(L, cand, acc, uR, tau, method="bruteforce"):
    ref = O.joint_replay(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, cand, acc, method=method)
    assert_scores_close(uR, ref, "union_R")
    for t, (a, r) in enumerate(zip(acc, ref)):
        if abs(r - tau) <= REL_TOL * tau:
            continue
        assert bool(a) == (r <= tau), f"step {t}: gpu {'accept' if a else 'reject'} but R_ref={r} tau={tau}"


@pytest.mark.parametrize("case,tau_mult", [("tiny", 1.5), ("tiny", 4.0), ("d128", 2.5)])
def test_joint_replay(ckv, case, tau_mult):
    """tau is a multiple of the smallest candidate effect, so the first
    candidate passes and the accumulated union later fails."""
    P, ctx = ckv
    w = WORKLOADS["tiny"] if case == "tiny" else scaled("q8b", n_tokens=5000, n_q_heads=8, n_kv_heads=2)
    L = make_layer(w, seed=21)
    dl = LayerOnDevice(L)
    kv, win, pages, m = _post_measure(P, ctx, dl)
    # candidates: the 40% of pages with the smallest post effect, forced
    R = m["R"].cpu().numpy()
    force = np.zeros(len(R), np.uint8)
    force[np.argsort(R, kind="stable")[: int(0.4 * len(R))]] = 1
    tau = float(tau_mult * R[force == 1].min())
    print(f"[joint] case={case} tau={tau:.4g} pages={len(L.pages)}", flush=True)
    zeros = torch.zeros_like(m["R"])
    cl = P.ckv_classify_pages(ctx, zeros, m["R"], force=torch.tensor(force).cuda())
    max_cand = int(force.sum()) + 3
    out = P.ckv_joint_test(ctx, kv, win, m["o"], m["lse"], pages, cl["cand"], cl["n_cand"], max_cand, tau)
    torch.cuda.synchronize()
    nc = int(cl["n_cand"].item())
    cand = cl["cand"].cpu().numpy()[:nc]
    acc = out["accepted"].cpu().numpy()
    uR = out["union_R"].cpu().numpy()
    assert np.all(acc[nc:] == 0) and np.all(np.isnan(uR[nc:]))
    assert int(out["n_accepted"].item()) == int(acc.sum())
    print(f"[joint] accepted {acc.sum()} of {nc}")
    assert 0 < acc.sum() < nc        # the case exercises both outcomes
    _check_replay(L, cand, acc[:nc], uR[:nc], tau, method="closed" if case == "d128" else "bruteforce")


def test_two_small_pages(ckv):
    """Uniform attention (Q = 0) over 400 tokens; two 4-token pages whose
    values differ, each alone below tau, together above (mean identity)."""
    P, ctx = ckv
    S, d = 400, 64
    k = np.zeros((1, S, d), np.float32)
    v = np.zeros((1, S, d), np.float32)
    v[0, :, 0] = 1.0
    v[0, 100:104, 1] = 0.8125        # exact in bf16
    v[0, 200:204, 1] = 0.8125
    q = np.zeros((1, 3, d), np.float32)
    pos = np.arange(S, dtype=np.int32)
    qpos = np.array([S, S + 1, S + 2], np.int32)
    pages = [(100, 4), (200, 4), (300, 4)]
    kb, vb, qb = dev_bf16(bf16_bits(k)), dev_bf16(bf16_bits(v)), dev_bf16(bf16_bits(q))
    kv = P.kv_view(kb, vb, dev_i32(pos))
    win = P.window_view(qb, dev_i32(qpos))
    pl = P.Pages([p[0] for p in pages], [p[1] for p in pages])
    m = P.ckv_measure_page_effects(ctx, kv, win, pl, want=("R", "o", "lse"))
    cand = torch.tensor([0, 1, 2], dtype=torch.int32, device="cuda")
    ncand = torch.tensor([3], dtype=torch.int32, device="cuda")
    out = P.ckv_joint_test(ctx, kv, win, m["o"], m["lse"], pl, cand, ncand, 3, 0.01)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out["accepted"].cpu().numpy(), [1, 0, 1])
    Vf = v[0].astype(np.float64)
    m1 = np.zeros(S, bool); m1[100:104] = True
    m2 = np.zeros(S, bool); m2[200:204] = True
    m3 = np.zeros(S, bool); m3[300:304] = True

    def ident(mask):
        n = S
        return (mask.sum() / n) * np.linalg.norm(Vf[mask].mean(0) - Vf[~mask].mean(0)) / np.linalg.norm(Vf.mean(0))
    want = [ident(m1), ident(m1 | m2), ident(m1 | m3)]
    assert_scores_close(out["union_R"].cpu().numpy(), want, "union_R")


def test_no_candidates(ckv):
    P, ctx = ckv
    L = make_layer(WORKLOADS["tiny"], seed=3)
    dl = LayerOnDevice(L)
    kv, win, pages, m = _post_measure(P, ctx, dl)
    cand = torch.full((5,), -1, dtype=torch.int32, device="cuda")
    ncand = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = P.ckv_joint_test(ctx, kv, win, m["o"], m["lse"], pages, cand, ncand, 5, 0.01)
    torch.cuda.synchronize()
    assert int(out["n_accepted"].item()) == 0 and out["accepted"].sum().item() == 0


def test_stress_forced_pages_small(ckv):
    """The stress construction at reduced size: forced pages fed in (R+ asc,
    R- desc, index asc) order, capped at 64, decisions replayed exactly."""
    P, ctx = ckv
    w = scaled("stress", n_tokens=4096, n_q_heads=8, n_kv_heads=2, max_cand=64)
    L = make_layer(w, seed=5)
    dl = LayerOnDevice(L)
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    Rm = P.ckv_measure_page_effects(ctx, P.kv_view(dl.k, dl.v, dl.pos, L.layout.s_pre),
                                    P.window_view(dl.q_pre, dl.qpos_pre), pages)["R"]
    kv, win, _, m = _post_measure(P, ctx, dl)
    cl = P.ckv_classify_pages(ctx, Rm, m["R"], force=torch.tensor(L.forced.astype(np.uint8)).cuda(),
                              max_cand=64)
    out = P.ckv_joint_test(ctx, kv, win, m["o"], m["lse"], pages, cl["cand"], cl["n_cand"], 64, 0.01)
    torch.cuda.synchronize()
    nc = int(cl["n_cand"].item())
    cand = cl["cand"].cpu().numpy()[:nc]
    acc = out["accepted"].cpu().numpy()[:nc]
    uR = out["union_R"].cpu().numpy()[:nc]
    print(f"[joint] stress: {acc.sum()} of {nc} accepted")
    _check_replay(L, cand, acc, uR, 0.01, method="closed")


def _dominant_union_layer(seed=31):
    """One KV head shared by 4 query heads (d 128, 1536 tokens, 8 window rows,
    32 pages of 32 tokens).  Page 3's keys follow query row (head 0, row 0),
    so that page alone carries > 0.99 of the row's mass; pages 10 and 11
    follow row (head 1, row 2) so that each carries just under half of it and
    their union > 0.9 (Eq. (6) is ill-conditioned there)."""
    rng = np.random.default_rng(seed)
    S, d, Hq, W = 1536, 128, 4, 8
    q = bf16_bits(rng.standard_normal((Hq, W, d)).astype(np.float32))
    qf = O.as_f64(q)
    k = rng.standard_normal((1, S, d))
    k[0, 352:384] = qf[0, 0] + 0.05 * rng.standard_normal((32, d))
    k[0, 576:640] = 0.57 * qf[1, 2] + 0.05 * rng.standard_normal((64, d))
    v = rng.standard_normal((1, S, d))
    kb, vb = bf16_bits(k.astype(np.float32)), bf16_bits(v.astype(np.float32))
    pos = np.arange(S, dtype=np.int32)
    qpos = np.arange(S, S + W, dtype=np.int32)
    pages = [(256 + 32 * i, 32) for i in range(32)]
    return kb, vb, q, pos, qpos, pages


def _union_mass(kb, vb, q, pos, qpos, pages, members, h, p):
    K, V, Q = O.as_f64(kb), O.as_f64(vb), O.as_f64(q)
    s = O.head_logits(Q[h], K[0], 1 / np.sqrt(K.shape[2]))
    a, _ = O.attend(s, O.visibility(pos, qpos), V[0])
    return float(sum(a[p, st:st + ln].sum() for st, ln in (pages[j] for j in members)))


@pytest.mark.parametrize("order,tau", [([10, 3, 11, 0, 1, 5], 1e30), ([0, 3, 1, 10, 11, 2, 4], 0.5),
                                       ([3, 10, 11, 6], 1e30)])
def test_joint_dominant_union(ckv, order, tau):
    """Unions whose mass in some row exceeds 0.9 (a dominant candidate with
    A > 0.99, and two pages of about 0.47 each) are recomputed by definition
    (Eq. (6) through the output without the union); every union effect is
    replayed by brute force at 2e-3 and every decision checked."""
    P, ctx = ckv
    kb, vb, q, pos, qpos, pages = _dominant_union_layer()
    # the construction does what it says (oracle, fp64)
    assert _union_mass(kb, vb, q, pos, qpos, pages, [3], 0, 0) > 0.99
    a10 = _union_mass(kb, vb, q, pos, qpos, pages, [10], 1, 2)
    a_pair = _union_mass(kb, vb, q, pos, qpos, pages, [10, 11], 1, 2)
    assert a10 < 0.9 < a_pair, (a10, a_pair)
    print(f"[joint] dominant union: order={order} tau={tau} A(10)={a10:.4f} A(10,11)={a_pair:.4f}", flush=True)
    kv = P.kv_view(dev_bf16(kb), dev_bf16(vb), dev_i32(pos))
    win = P.window_view(dev_bf16(q), dev_i32(qpos))
    pl = P.Pages([p[0] for p in pages], [p[1] for p in pages])
    m = P.ckv_measure_page_effects(ctx, kv, win, pl, want=("R", "o", "lse"))
    cand = torch.tensor(order, dtype=torch.int32, device="cuda")
    ncand = torch.tensor([len(order)], dtype=torch.int32, device="cuda")
    out = P.ckv_joint_test(ctx, kv, win, m["o"], m["lse"], pl, cand, ncand, len(order), tau)
    torch.cuda.synchronize()
    acc = out["accepted"].cpu().numpy()
    uR = out["union_R"].cpu().numpy()
    assert int(out["n_accepted"].item()) == int(acc.sum())
    print(f"[joint] accepted {acc.astype(int).tolist()} union_R {np.round(uR, 4).tolist()}", flush=True)
    ref = O.joint_replay(kb, vb, pos, q, qpos, pages, order, acc, method="bruteforce")
    assert_scores_close(uR, ref, "union_R (dominant unions)")
    for t, (a, r) in enumerate(zip(acc, ref)):
        if abs(r - tau) <= REL_TOL * tau:
            continue
        assert bool(a) == (r <= tau), f"step {t}: gpu {'accept' if a else 'reject'} but R_ref={r} tau={tau}"
