"""Plant plausible mistakes in the oracle (on the CPU) and check that a pin fails.

Each mutant replaces one oracle function for the duration of a test; the
check that follows is the same comparison a pin in test_oracle_pins makes.
"""
import math

import numpy as np
import pytest

import oracle as O
import oracle.commitkv_oracle as OM
from tests.test_oracle_pins import _random_case, _two_small_pages


def _closed_no_renorm(a, o, v, delete, vis):
    """Mutant: forgets the 1/(1 - A) of Eq. (6)."""
    sel = vis & delete[None, :]
    a_e = np.where(sel, a, 0.0)
    A = a_e.sum(axis=1)
    u = a_e @ v
    return np.linalg.norm(u - A[:, None] * o, axis=1) / np.linalg.norm(o, axis=1)


def _closed_sign_flip(a, o, v, delete, vis):
    """Mutant: u + A o instead of u - A o."""
    sel = vis & delete[None, :]
    a_e = np.where(sel, a, 0.0)
    A = a_e.sum(axis=1)
    u = a_e @ v
    return np.linalg.norm(u + A[:, None] * o, axis=1) / ((1 - A) * np.linalg.norm(o, axis=1))


@pytest.mark.parametrize("mutant", [_closed_no_renorm, _closed_sign_flip])
def test_closed_form_mutants_are_caught(monkeypatch, mutant):
    K, V, Q, pos, qpos, pages = _random_case(0)
    Rb, _ = O.page_effects(K, V, pos, Q, qpos, pages, method="bruteforce")
    monkeypatch.setattr(OM, "deletion_ratio_closed_form", mutant)
    with np.errstate(all="ignore"):
        Rc, _ = OM.page_effects(K, V, pos, Q, qpos, pages, method="closed")
    fin = np.isfinite(Rb) & np.isfinite(Rc)
    assert not np.allclose(Rc[fin], Rb[fin], rtol=1e-10)


def test_visibility_off_by_one_is_caught(monkeypatch):
    """Mutant: strict p_i < p drops the window row's own token."""
    monkeypatch.setattr(OM, "visibility",
                        lambda pos, qpos: np.asarray(pos)[None, :] < np.asarray(qpos)[:, None])
    K = np.array([[[0.0, 0.0], [math.log(3.0), 0.0]]])
    V = np.array([[[1.0, 0.0], [0.0, 1.0]]])
    Q = np.array([[[1.0, 0.0]]])
    R, _ = OM.page_effects(K, V, np.array([0, 1]), Q, np.array([1]), [(1, 1)], scale=1.0)
    assert R[0] != pytest.approx(3 / math.sqrt(5))


def test_percentile_non_strict_is_caught(monkeypatch):
    def mutant(R):
        R = np.asarray(R, float)
        n = R.size
        return np.array([((R <= R[j]).sum() - 1) / (n - 1) for j in range(n)])
    monkeypatch.setattr(OM, "percentile_ranks", mutant)
    assert not np.array_equal(OM.percentile_ranks([0.1, 0.1, 0.2]), [0.0, 0.0, 1.0])


def test_lifecycle_swap_is_caught(monkeypatch):
    """Mutant: candidate defined as L- and H+ (the transition reversed)."""
    def mutant(H_pre, L_pre, H_post, L_post, precommit=True):
        lam = np.full(len(H_pre), O.UNCERTAIN, np.uint8)
        lam[L_pre & H_post] = O.CANDIDATE
        lam[L_pre & L_post] = O.DORMANT
        lam[H_pre & L_post] = O.NEWLY_ACTIVE
        lam[H_pre & H_post] = O.STILL_ACTIVE
        return lam
    monkeypatch.setattr(OM, "lifecycle", mutant)
    lam, *_ = OM.classify([0.9, 0.05, 0.001, 0.01, 0.03], [0.05, 0.01, 0.002, 0.5, 0.04],
                          starts=[0, 16, 32, 48, 64])
    assert lam[1] != O.CANDIDATE


def test_joint_without_union_is_caught(monkeypatch):
    """Mutant: tests each candidate alone instead of A u {E} (Eq. (11))."""
    K, V, Q, pos, qpos, pages = _two_small_pages()
    real = OM.union_effect
    monkeypatch.setattr(OM, "union_effect",
                        lambda K, V, pos, Q, qpos, pages, members, scale=None, method="bruteforce":
                        real(K, V, pos, Q, qpos, pages, members[-1:], scale, method))
    acc, _ = OM.joint_test(K, V, pos, Q, qpos, pages, [0, 1, 2], tau_joint=0.01)
    assert not np.array_equal(acc, [True, False, True])


def test_protect_skip_instead_of_stop_is_caught(monkeypatch):
    def mutant(starts, lens, R_pre, B, eta=0.125, max_pages=16):
        BN = int(math.floor(eta * B))
        order = sorted(range(len(starts)), key=lambda j: (-R_pre[j], starts[j]))
        taken, tok = [], 0
        for j in order:
            if len(taken) < max_pages and tok + lens[j] <= BN:
                taken.append(j)
                tok += lens[j]
        return np.array(taken)
    monkeypatch.setattr(OM, "protect_pending", mutant)
    got = OM.protect_pending([0, 4, 8, 10, 14], [4, 4, 2, 4, 1], [0.5, 0.9, 0.7, 0.7, 0.1], 64)
    assert not np.array_equal(got, [1, 2])


# ---------------------------------------------------------------- lifecycle driver (Algorithm 1)
def test_driver_scan_cap_oldest_is_caught(monkeypatch):
    """Mutant: the scan cap keeps the oldest pages instead of the newest."""
    import oracle.lifecycle as OL
    from tests.test_oracle_lifecycle import CALL, OBS, _push
    real = OL.Agent.eligible

    def mutant(self):
        cap, self.max_scan = self.max_scan, 0
        pages = real(self)
        self.max_scan = cap
        return pages[:cap]
    monkeypatch.setattr(OL.Agent, "eligible", mutant)
    a = OL.Agent(1, 1, 2, page_size=4, budget=1000, max_scan_pages=2)
    p = _push(a, CALL, 0, [[0, 0]] * 12, [[1, 0]] * 12)
    _push(a, OBS, p, [[0, 0]] * 6, [[1, 0]] * 6)
    assert a.eligible() != [(12, 4), (16, 2)]


def test_driver_checkpoint_keeping_retired_is_caught(monkeypatch):
    """Mutant: a checkpoint under the budget skips compaction even though a
    retired page is resident (the hand-built page then stays)."""
    import math
    import oracle.lifecycle as OL
    from tests.test_oracle_lifecycle import _hand_episode
    real = OL.Agent.checkpoint

    def mutant(self, Q, qpos, score=None):
        if self.pos.size <= self.B:
            return dict(compacted=False)
        return real(self, Q, qpos, score)
    monkeypatch.setattr(OL.Agent, "checkpoint", mutant)
    a, _ = _hand_episode()
    q_post = np.array([[[-2000 * math.sqrt(2.0)] * 2] * 2])
    a.post(q_post, np.array([48, 49]))
    a.checkpoint(q_post, np.array([48, 49]))
    assert np.isin(np.arange(16, 20), a.pos).any()      # the pin's expectation fails


def test_driver_protecting_partial_pages_is_caught(monkeypatch):
    """Mutant: pending pages that lost tokens are still offered for protection."""
    import oracle.lifecycle as OL
    from tests.test_oracle_lifecycle import _hand_episode

    def mutant(self):
        pend, r = list(self.pending[0]), np.asarray(self.pending[1], np.float64)
        return pend, r, []
    monkeypatch.setattr(OL.Agent, "checkpoint_lists", mutant)
    a, rep = _hand_episode()
    a.B = 32
    score = np.zeros(a.pos.size, np.float32)
    score[:32] = 1.0
    a.checkpoint(None, None, score=score)
    lost = [p for p in rep["pages"] if not a.fully_resident(p)]
    assert any(p in a.checkpoint_lists()[0] for p in lost)
