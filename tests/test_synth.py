"""The seeded input generator: layouts, pages and windows match the stated recipe."""
import numpy as np
import pytest

from synth import WORKLOADS, bf16_bits, bf16_bits_to_f32, make_layer, make_layout, scaled
from synth.workloads import OBSERVATION, REASONING, TOOL_CALL, rng_for


@pytest.mark.parametrize("name", ["tiny", "q8b", "q32b", "stress"])
def test_layout_invariants(name):
    w = WORKLOADS[name]
    lay = make_layout(w, rng_for(w, 0, 0, 0, 0))
    ev = lay.events
    assert ev[0][1] == 0 and sum(e[2] for e in ev) == w.n_tokens
    for (k0, s0, l0), (k1, s1, l1) in zip(ev, ev[1:]):
        assert s0 + l0 == s1
    # commit tail: tool call (>= W), 128-token observation, W-token window
    assert ev[-3][0] == TOOL_CALL and ev[-3][2] >= w.window
    assert ev[-2][0] == OBSERVATION and ev[-2][2] == w.obs_len
    assert ev[-1][0] == REASONING and ev[-1][2] == w.window
    assert lay.s_pre == ev[-3][1] + ev[-3][2]
    # pages: sorted, disjoint, <= G, inside one tool-call/observation event, before s_pre
    st, ln = lay.page_start, lay.page_len
    assert np.all(np.diff(st) > 0) and np.all(st[:-1] + ln[:-1] <= st[1:])
    assert ln.min() >= 1 and ln.max() <= w.page_size
    assert st[-1] + ln[-1] <= lay.s_pre
    bounds = [(s, s + l) for k, s, l in ev if k != REASONING]
    for a, b in zip(st, st + ln):
        assert any(lo <= a and b <= hi for lo, hi in bounds)
    assert len(lay.pending_idx) == -(-ev[-3][2] // w.page_size)
    np.testing.assert_array_equal(lay.qrows_pre, np.arange(lay.s_pre - w.window, lay.s_pre))
    np.testing.assert_array_equal(lay.qrows_post, np.arange(w.n_tokens - w.window, w.n_tokens))


def test_seeded_and_heavy_hitters():
    w = WORKLOADS["tiny"]
    a, b = make_layer(w, seed=3), make_layer(w, seed=3)
    assert np.array_equal(a.k, b.k) and np.array_equal(a.q_post, b.q_post)
    c = make_layer(w, seed=4)
    assert not np.array_equal(a.k, c.k)
    kf = bf16_bits_to_f32(a.k)
    big = np.abs(kf).max(axis=2).max(axis=0)
    n_heavy = int(round(w.heavy_frac * w.n_tokens))
    assert (big > 6).sum() >= n_heavy * 0.8


def test_bf16_rounding_is_nearest_even():
    import torch
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, -2.5, 3.0e38], np.float32)
    got = bf16_bits_to_f32(bf16_bits(x))
    np.testing.assert_array_equal(got[:4], np.array([1.0, 1.0, 1.0 + 2**-6, -2.5], np.float32))
    x = np.random.default_rng(0).standard_normal(10000).astype(np.float32) * 100
    want = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(bf16_bits_to_f32(bf16_bits(x)), want)


def test_gapped_positions_and_stress_forcing():
    w = scaled("tiny", gapped_positions=True)
    L = make_layer(w)
    assert np.all(np.diff(L.pos) >= 1) and L.pos[-1] > w.n_tokens
    np.testing.assert_array_equal(L.qpos_post, L.pos[-w.window:])
    s = make_layer(scaled("stress", n_tokens=4096, n_kv_heads=2, n_q_heads=4))
    assert 0.25 < s.forced.mean() < 0.35
    kf = bf16_bits_to_f32(s.k[:, :, 0])
    for j in np.flatnonzero(s.forced)[:5]:
        st, ln = s.layout.page_start[j], s.layout.page_len[j]
        assert np.all(kf[:, st:st + ln] > 11)
    assert np.count_nonzero(kf) == s.forced @ s.layout.page_len * 2
