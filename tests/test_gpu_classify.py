"""GPU parity of ckv_classify_pages (Sec. 3.2, Eq. (8)-(10); candidate order of Sec. 3.3).

Given the same float32 effects, lifecycle states, percentiles and the ordered
candidate list must be identical to the oracle's (thresholds rounded to
float32 on both sides).  Given each side's own measured effects, states may
differ only for pages whose effect or percentile sits within the score
tolerance of a threshold.
"""
import numpy as np
import pytest
import torch

import oracle as O
from synth import WORKLOADS, make_layer, scaled
from tests.gpu_util import LayerOnDevice, REL_TOL, oracle_pass

pytestmark = pytest.mark.gpu

TH = dict(tau_use=0.05, tau_dead=0.01, rho_use=0.75, rho_dead=0.25)
TH32 = {k: float(np.float32(v)) for k, v in TH.items()}


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _gpu_classify(P, ctx, Rm, Rp, force=None, max_cand=0, th=None):
    Rm_t = torch.tensor(np.asarray(Rm, np.float32)).cuda()
    Rp_t = torch.tensor(np.asarray(Rp, np.float32)).cuda()
    f = None if force is None else torch.tensor(np.asarray(force, np.uint8)).cuda()
    out = P.ckv_classify_pages(ctx, Rm_t, Rp_t, th or TH, force=f, max_cand=max_cand)
    torch.cuda.synchronize()
    n_cand = int(out["n_cand"].item())
    return (out["lam"].cpu().numpy(), out["P_pre"].cpu().numpy(), out["P_post"].cpu().numpy(),
            out["cand"].cpu().numpy()[:n_cand], n_cand, out["cand"].cpu().numpy())


def _oracle(Rm, Rp, max_cand=None):
    Rm = np.asarray(Rm, np.float32).astype(np.float64)
    Rp = np.asarray(Rp, np.float32).astype(np.float64)
    return O.classify(Rm, Rp, np.arange(len(Rm)), max_cand=max_cand, **TH32)


def test_hand_table(ckv):
    P, ctx = ckv
    Rm = [0.9, 0.05, 0.001, 0.01, 0.03]
    Rp = [0.05, 0.01, 0.002, 0.5, 0.04]
    lam, Pm, Pp, cand, n, _ = _gpu_classify(P, ctx, Rm, Rp)
    np.testing.assert_array_equal(lam, [O.STILL_ACTIVE, O.CANDIDATE, O.DORMANT, O.NEWLY_ACTIVE, O.UNCERTAIN])
    np.testing.assert_array_equal(Pm, [1.0, 0.75, 0.0, 0.25, 0.5])
    np.testing.assert_array_equal(cand, [1])


@pytest.mark.parametrize("n", [1, 2, 5, 257, 700, 2600])
def test_random_effects_identical(ckv, n):
    P, ctx = ckv
    r = np.random.default_rng(n)
    # log-uniform effects around the thresholds, with ties
    Rm = np.exp(r.uniform(np.log(1e-4), np.log(2.0), n)).astype(np.float32)
    Rp = np.exp(r.uniform(np.log(1e-4), np.log(2.0), n)).astype(np.float32)
    Rm[r.choice(n, n // 5)] = 0.01
    Rp[r.choice(n, n // 5)] = np.float32(0.05)
    Rp[r.choice(n, n // 7)] = np.float32(0.003)
    lam, Pm, Pp, cand, nc, raw = _gpu_classify(P, ctx, Rm, Rp)
    lam_o, Pm_o, Pp_o, cand_o = _oracle(Rm, Rp)
    np.testing.assert_array_equal(lam, lam_o)
    np.testing.assert_allclose(Pm, Pm_o, rtol=1e-7)
    np.testing.assert_allclose(Pp, Pp_o, rtol=1e-7)
    np.testing.assert_array_equal(cand, cand_o)
    assert np.all(raw[nc:] == -1)


@pytest.mark.parametrize("n", [300, 1500])
def test_infinite_effects(ckv, n):
    """Pages that hold every visible token have R = +inf (Eq. (6)-(7)):
    they rank above every finite page and tie with each other; zero
    effects tie at the bottom."""
    P, ctx = ckv
    r = np.random.default_rng(n + 1)
    Rm = np.exp(r.uniform(np.log(1e-4), np.log(2.0), n)).astype(np.float32)
    Rp = np.exp(r.uniform(np.log(1e-4), np.log(2.0), n)).astype(np.float32)
    Rm[::37] = np.inf
    Rp[::41] = np.inf
    Rp[5::53] = 0.0
    lam, Pm, Pp, cand, nc, raw = _gpu_classify(P, ctx, Rm, Rp)
    lam_o, Pm_o, Pp_o, cand_o = _oracle(Rm, Rp)
    np.testing.assert_array_equal(lam, lam_o)
    np.testing.assert_allclose(Pm, Pm_o, rtol=1e-7)
    np.testing.assert_allclose(Pp, Pp_o, rtol=1e-7)
    np.testing.assert_array_equal(cand, cand_o)
    assert np.all(raw[nc:] == -1)


def test_force_and_cap(ckv):
    P, ctx = ckv
    r = np.random.default_rng(0)
    n = 300
    Rm = r.uniform(0, 1, n).astype(np.float32)
    Rp = r.uniform(0, 1, n).astype(np.float32)
    Rp[:20] = Rp[20:40]            # ties in R+ resolved by R- then index
    force = np.zeros(n, np.uint8)
    force[r.choice(n, 90, replace=False)] = 1
    lam, _, _, cand, nc, _ = _gpu_classify(P, ctx, Rm, Rp, force=force, max_cand=64)
    lam_o, *_ = _oracle(Rm, Rp)
    members = [j for j in range(n) if force[j] or lam_o[j] == O.CANDIDATE]
    members.sort(key=lambda j: (float(Rp[j]), -float(Rm[j]), j))
    np.testing.assert_array_equal(cand, members[:64])
    assert nc == 64


def test_empty(ckv):
    P, ctx = ckv
    out = P.ckv_classify_pages(ctx, torch.zeros(0, device="cuda"), torch.zeros(0, device="cuda"), TH)
    torch.cuda.synchronize()
    assert int(out["n_cand"].item()) == 0


def _excused(R_ref_pre, R_ref_post, rel=REL_TOL):
    """Pages whose state may legitimately differ: an effect within rel of a
    tau, or a rho inside the percentile band obtained by treating every
    comparison within rel as ambiguous."""
    n = len(R_ref_pre)
    ex = np.zeros(n, bool)
    for R in (R_ref_pre, R_ref_post):
        for tau in (TH["tau_use"], TH["tau_dead"]):
            ex |= np.abs(R - tau) <= rel * tau
        if n > 1:
            lo = np.array([(R < R[j] * (1 - 2 * rel)).sum() for j in range(n)]) / (n - 1)
            hi = np.array([((R < R[j] * (1 + 2 * rel)).sum() - 1) for j in range(n)]) / (n - 1)
            for rho in (TH["rho_use"], TH["rho_dead"]):
                ex |= (lo <= rho) & (rho <= hi)
    return ex


@pytest.mark.parametrize("case", ["tiny", "d128"])
def test_states_from_measured_effects(ckv, case):
    P, ctx = ckv
    w = WORKLOADS["tiny"] if case == "tiny" else scaled("q8b", n_tokens=6000, n_q_heads=8, n_kv_heads=2)
    L = make_layer(w, seed=11)
    dl = LayerOnDevice(L)
    pages = P.Pages(L.layout.page_start, L.layout.page_len)
    Rm_g = P.ckv_measure_page_effects(ctx, P.kv_view(dl.k, dl.v, dl.pos, L.layout.s_pre),
                                      P.window_view(dl.q_pre, dl.qpos_pre), pages)["R"]
    Rp_g = P.ckv_measure_page_effects(ctx, P.kv_view(dl.k, dl.v, dl.pos),
                                      P.window_view(dl.q_post, dl.qpos_post), pages)["R"]
    out = P.ckv_classify_pages(ctx, Rm_g, Rp_g, TH)
    torch.cuda.synchronize()
    lam = out["lam"].cpu().numpy()
    Rm_o, _ = oracle_pass(L, "pre")
    Rp_o, _ = oracle_pass(L, "post")
    lam_o, *_ = O.classify(Rm_o, Rp_o, L.layout.page_start, **TH)
    ex = _excused(Rm_o, Rp_o)
    diff = np.flatnonzero((lam != lam_o) & ~ex)
    assert diff.size == 0, f"states differ at {diff[:10]}: gpu {lam[diff[:10]]} oracle {lam_o[diff[:10]]}"
    print(f"[classify] {case}: states {np.bincount(lam, minlength=5)}; excused {ex.sum()}")
