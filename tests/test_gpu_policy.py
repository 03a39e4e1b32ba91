"""GPU parity of the Sec. 4.4 ablation switches (ckv_set_policy) for the
classification and the joint test; the selection variants sit with the other
selection cases in test_gpu_select.

Bar as for the complete method: identical states, percentiles and candidate
lists given the same float32 effects; the joint test's accepted flags exact
and union_R within the score tolerance of the closed-form mean identity.
"""
import numpy as np
import pytest
import torch

import oracle as O
from synth import bf16_bits
from tests.gpu_util import assert_scores_close, dev_bf16, dev_i32

pytestmark = pytest.mark.gpu

TH = dict(tau_use=0.05, tau_dead=0.01, rho_use=0.75, rho_dead=0.25)
TH32 = {k: float(np.float32(v)) for k, v in TH.items()}


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _classify(P, ctx, Rm, Rp, ablation):
    ctx.set_policy(*ablation)
    try:
        out = P.ckv_classify_pages(ctx, torch.tensor(np.asarray(Rm, np.float32)).cuda(),
                                   torch.tensor(np.asarray(Rp, np.float32)).cuda(), TH)
    finally:
        ctx.set_policy()
    torch.cuda.synchronize()
    nc = int(out["n_cand"].item())
    return (out["lam"].cpu().numpy(), out["P_pre"].cpu().numpy(), out["P_post"].cpu().numpy(),
            out["cand"].cpu().numpy()[:nc])


def test_set_and_get(ckv):
    P, ctx = ckv
    ctx.set_policy("no_joint", "no_percentile")
    assert ctx.policy() == 4 | 2
    ctx.set_policy()
    assert ctx.policy() == 0
    with pytest.raises(P.CKVError):
        ctx.check(ctx._lib.ckv_set_policy(ctx.handle, 1 << 7))
    assert ctx.policy() == 0


def test_hand_table(ckv):
    """The five-page table of the lifecycle pins under each classification
    switch: without the pre-commit state the dormant page (L-, L+) becomes a
    candidate too; without percentiles the page with R- = 0.05 (percentile
    0.75) is high by its absolute effect alone either way, and the page with
    R+ = 0.04 stays uncertain."""
    P, ctx = ckv
    Rm = [0.9, 0.05, 0.001, 0.01, 0.03]
    Rp = [0.05, 0.01, 0.002, 0.5, 0.04]
    lam, *_, cand = _classify(P, ctx, Rm, Rp, ("no_precommit",))
    np.testing.assert_array_equal(lam, [O.STILL_ACTIVE, O.CANDIDATE, O.CANDIDATE, O.NEWLY_ACTIVE,
                                        O.UNCERTAIN])
    np.testing.assert_array_equal(cand, [2, 1])
    lam, *_, cand = _classify(P, ctx, Rm, Rp, ("no_lifecycle",))
    np.testing.assert_array_equal(lam, [O.STILL_ACTIVE, O.CANDIDATE, O.DORMANT, O.NEWLY_ACTIVE,
                                        O.UNCERTAIN])
    assert cand.size == 0


@pytest.mark.parametrize("ablation", [("no_precommit",), ("no_percentile",), ("no_lifecycle",),
                                      ("no_precommit", "no_percentile")])
@pytest.mark.parametrize("n", [1, 5, 700, 2600])
def test_random_effects_identical(ckv, ablation, n):
    P, ctx = ckv
    r = np.random.default_rng(100 + n)
    Rm = np.exp(r.uniform(np.log(1e-4), np.log(2.0), n)).astype(np.float32)
    Rp = np.exp(r.uniform(np.log(1e-4), np.log(2.0), n)).astype(np.float32)
    Rm[r.choice(n, n // 5)] = 0.01
    Rp[r.choice(n, n // 5)] = np.float32(0.05)
    lam, Pm, Pp, cand = _classify(P, ctx, Rm, Rp, ablation)
    lam_o, Pm_o, Pp_o, cand_o = O.classify(Rm.astype(np.float64), Rp.astype(np.float64),
                                           np.arange(n), ablation=ablation, **TH32)
    np.testing.assert_array_equal(lam, lam_o)
    np.testing.assert_allclose(Pm, Pm_o, rtol=1e-7)
    np.testing.assert_allclose(Pp, Pp_o, rtol=1e-7)
    np.testing.assert_array_equal(cand, cand_o)


def test_no_joint_accepts_every_candidate(ckv):
    """Two 4-token pages each below tau alone and above it together (uniform
    attention, so the union effect is the mean identity): the complete method
    rejects the second, the variant without the Eq. (11) gate accepts all
    three and reports the effect of each growing union."""
    P, ctx = ckv
    S, d = 400, 64
    k = np.zeros((1, S, d), np.float32)
    v = np.zeros((1, S, d), np.float32)
    v[0, :, 0] = 1.0
    v[0, 100:104, 1] = 0.8125
    v[0, 200:204, 1] = 0.8125
    q = np.zeros((1, 3, d), np.float32)
    pos = np.arange(S, dtype=np.int32)
    qpos = np.array([S, S + 1, S + 2], np.int32)
    pages = [(100, 4), (200, 4), (300, 4)]
    kv = P.kv_view(dev_bf16(bf16_bits(k)), dev_bf16(bf16_bits(v)), dev_i32(pos))
    win = P.window_view(dev_bf16(bf16_bits(q)), dev_i32(qpos))
    pl = P.Pages([p[0] for p in pages], [p[1] for p in pages])
    m = P.ckv_measure_page_effects(ctx, kv, win, pl, want=("R", "o", "lse"))
    cand = torch.tensor([0, 1, 2], dtype=torch.int32, device="cuda")
    ncand = torch.tensor([3], dtype=torch.int32, device="cuda")
    ctx.set_policy("no_joint")
    try:
        out = P.ckv_joint_test(ctx, kv, win, m["o"], m["lse"], pl, cand, ncand, 3, 0.01)
    finally:
        ctx.set_policy()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out["accepted"].cpu().numpy(), [1, 1, 1])
    assert int(out["n_accepted"].item()) == 3
    Vf = v[0].astype(np.float64)
    masks = [np.zeros(S, bool) for _ in pages]
    for mk, (s0, ln) in zip(masks, pages):
        mk[s0:s0 + ln] = True

    def ident(mask):
        return (mask.sum() / S) * np.linalg.norm(Vf[mask].mean(0) - Vf[~mask].mean(0)) \
            / np.linalg.norm(Vf.mean(0))
    want = [ident(masks[0]), ident(masks[0] | masks[1]), ident(masks[0] | masks[1] | masks[2])]
    assert_scores_close(out["union_R"].cpu().numpy(), want, "union_R")
    # the oracle's variant on the same inputs (exact in bf16) takes the same decisions
    acc_o, ur_o = O.joint_test(k, v, pos, q, qpos, pages, [0, 1, 2], tau_joint=0.01, gate=False)
    np.testing.assert_array_equal(acc_o, [True, True, True])
    assert_scores_close(out["union_R"].cpu().numpy(), ur_o, "union_R vs oracle")
