"""Pins of the lifecycle driver oracle (Algorithm 1; oracle/lifecycle.py).

Each pin checks the driver against a hand-derived outcome or an invariant of
the paper, not against a re-run of itself: pages cut from event starts
(Sec. 3.1), the scan cap (Sec. 4.1), a hand-built high-to-low page retired
and removed while a dormant page stays (Eq. (10)-(11), Algorithm 1),
pending protection surviving a checkpoint (Eq. (12)-(13)), and, over a whole
synthetic episode, |I_j| <= B with the cache holding exactly the
trajectory's tokens at the resident positions (Eq. (4)).
"""
import math

import numpy as np

import oracle as O
from oracle.lifecycle import Agent
from synth.trajectory import TRAJECTORIES, kv_rows, make_trajectory, scaled_trajectory
from tests.agent_util import oracle_agent, run_oracle

PROMPT, REASON, CALL, OBS = 3, 0, 1, 2


def _tok(rows):
    """float rows -> [1 head, n, d] float64 (the oracle takes real arrays too)."""
    return np.asarray(rows, np.float64)[None]


def _push(agent, kind, p0, k, v):
    n = len(k)
    agent.append(kind, p0, p0 + n, [_tok(k)], [_tok(v)], decoded=kind in (REASON, CALL), begins_event=True)
    return p0 + n


def test_pages_cut_from_event_start():
    a = Agent(1, 1, 2, page_size=16, budget=1000)
    p = _push(a, PROMPT, 0, [[0, 0]] * 5, [[1, 0]] * 5)
    p = _push(a, CALL, p, [[0, 0]] * 40, [[1, 0]] * 40)
    p = _push(a, REASON, p, [[0, 0]] * 3, [[1, 0]] * 3)
    _push(a, OBS, p, [[0, 0]] * 17, [[1, 0]] * 17)
    assert a.agent_pages() == [(5, 16), (21, 16), (37, 8), (48, 16), (64, 1)]


def test_scan_cap_takes_the_most_recent_pages():
    a = Agent(1, 1, 2, page_size=4, budget=1000, max_scan_pages=2)
    p = _push(a, CALL, 0, [[0, 0]] * 12, [[1, 0]] * 12)
    _push(a, OBS, p, [[0, 0]] * 6, [[1, 0]] * 6)
    assert a.eligible() == [(12, 4), (16, 2)]
    a.retire([(16, 2)])
    assert a.eligible() == [(8, 4), (12, 4)]


def _hand_episode():
    """d = 2, one head, G = 4.  Keys (0, 0) everywhere except page A1 =
    positions 16..19 (keys (1, 0)) and page D = 24..27 (keys (0, 1)).
    Q- = (3 sqrt2, -2000 sqrt2): A1 carries most of the pre-commit mass, D
    none (its logit -2000 underflows).  Q+ = (-2000 sqrt2, -2000 sqrt2): A1
    and D are both unattended after the observation (R+ = 0 exactly), the
    other pages share uniform attention with distinct values (R+ > 0).
    So A1 is H- and L+ (a completion candidate whose union effect is 0) and D
    is L- and L+ (dormant)."""
    a = Agent(1, 1, 2, page_size=4, budget=64, keep_recent=0, method="bruteforce")
    z = [0.0, 0.0]
    p = _push(a, PROMPT, 0, [z] * 16, [[1, 0]] * 16)
    p = _push(a, CALL, p, [[1, 0]] * 4 + [z] * 4, [[0, 1]] * 4 + [[1, 2]] * 4)      # A1, X2
    p = _push(a, OBS, p, [[0, 1]] * 4 + [z] * 4, [[1, -1]] * 4 + [[1, -2]] * 4)    # D, Y2
    p = _push(a, REASON, p, [z] * 8, [[1, 0.5]] * 8)
    p = _push(a, CALL, p, [z] * 4, [[1, 3]] * 4)                                    # Z1
    assert p == 44
    s2 = math.sqrt(2.0)
    q_pre = np.array([[[3 * s2, -2000 * s2]] * 2])
    rep = a.commit(q_pre, np.array([42, 43]))
    assert rep["pages"] == [(16, 4), (20, 4), (24, 4), (28, 4), (40, 4)]
    p = _push(a, OBS, p, [z] * 4, [[1, -3]] * 4)
    p = _push(a, REASON, p, [z] * 2, [[1, 0]] * 2)
    return a, rep


def test_hand_built_transition_is_retired_and_removed():
    a, rep = _hand_episode()
    R_pre = rep["R_pre"]
    assert R_pre[2] == 0.0 and R_pre[0] == R_pre.max() and R_pre[0] >= 0.05
    q_post = np.array([[[-2000 * math.sqrt(2.0)] * 2] * 2])
    m = a.post(q_post, np.array([48, 49]))
    assert m["R_post"][0] == 0.0 and m["R_post"][2] == 0.0
    assert m["lam"][0] == O.CANDIDATE and m["lam"][2] == O.DORMANT
    assert a.retired == [(16, 4)]
    assert a.pending is None
    # a checkpoint under the budget still removes the retired page (and only it)
    c = a.checkpoint(q_post, np.array([48, 49]))
    assert c["compacted"]
    assert not np.isin(np.arange(16, 20), a.pos).any()
    assert np.isin(np.arange(24, 28), a.pos).all()
    assert a.pos.size == 46 and a.retired == []


def test_pending_protection_survives_a_checkpoint():
    """Between a commit and its post window, the pending pages of largest R-
    (at most 16 pages and B_N tokens) are kept whatever their score."""
    a, rep = _hand_episode()
    a.B = 32                                   # B_N = 4: exactly one page fits
    score = np.zeros(a.pos.size, np.float32)   # every free token scores the same
    score[:32] = 1.0                           # ... except a preferred prefix
    c = a.checkpoint(None, None, score=score)
    assert c["protected"] == [(16, 4)]          # largest R-
    assert np.isin(np.arange(16, 20), a.pos).all()
    assert a.pos.size == 32
    # a pending page that lost tokens is no longer protectable or measurable
    lost = [p for p in rep["pages"] if not a.fully_resident(p)]
    assert lost and all(p not in a.checkpoint_lists()[0] for p in lost)


def test_episode_invariants():
    cfg = TRAJECTORIES["tiny_agent"]
    traj = make_trajectory(cfg, seed=3, n_turns=6)
    agent = oracle_agent(cfg)
    seen = dict(checkpoint=0, compacted=0, post=0, commit=0, retired=0)

    def hook(act, rep):
        if act[0] == "append":
            return
        seen[act[0]] += 1
        if act[0] == "checkpoint" and rep["compacted"]:
            seen["compacted"] += 1
            assert agent.pos.size <= cfg.budget
            assert np.all(np.diff(agent.pos) > 0)
            for p in rep["protected"]:
                assert agent.fully_resident(p)
            assert agent.retired == []
            for l in range(cfg.n_layers):
                # Eq. (4): the cache holds exactly the trajectory's tokens at the kept positions
                k, v = kv_rows(traj, l, 0, traj.n_tokens)
                np.testing.assert_array_equal(agent.K[l], k[:, agent.pos])
                np.testing.assert_array_equal(agent.V[l], v[:, agent.pos])
        if act[0] == "post":
            seen["retired"] += int(np.sum(rep["accepted"]))
            assert set(np.flatnonzero(rep["lam"] == O.CANDIDATE)) <= set(rep["cand"].tolist())

    run_oracle(traj, agent, hook)
    assert seen["compacted"] >= 2 and seen["post"] >= 4 and seen["commit"] >= 5


def test_scaled_trajectory_and_schedule_shape():
    cfg = scaled_trajectory("paper_agent", n_layers=2)
    t = make_trajectory(cfg, seed=1, n_turns=3)
    kinds = [e[0] for e in t.events]
    assert kinds == [PROMPT, REASON, CALL, OBS, REASON, CALL, OBS, REASON, 4]
