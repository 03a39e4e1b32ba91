"""Seeded synthetic agent-cache workloads shared by the tests, the bench and smoke.

This module only draws inputs: event layouts, page spans, bf16 keys, values
and queries, positions and query-window positions.  It holds none of the
method's arithmetic (no attention, no deletion effect, no selection), so the
oracle and the HIP path can both consume its output without sharing code.

The workloads stand in for the paper's agent benchmarks (Sec. 4.1), which are
not available: a ReAct trajectory (Sec. 3.1, Eq. (1)) is laid out as a cycle
of reasoning, tool-call and observation events; tool calls and observations
are agent events cut into pages of at most G tokens (Sec. 3.1); the pre- and
post-commit windows follow Eq. (5).

Named workloads (sizes chosen to match the per-layer shapes of Qwen3-8B and
Qwen3-32B style models):

* ``tiny``   1 KV head shared by 4 query heads, d=64, 2048 cached tokens, 16-token
             pages over events of 32..256 tokens, 32-row windows, budget 1024.
* ``q8b``    8 KV heads / 32 query heads, d=128, 32768 tokens, 32-token pages
             over events of 64..2048 tokens, 64-row windows, budget 8192.
* ``q8b_stack`` the ``q8b`` layer over 36 layers x 4 sequences at 65536 tokens,
             budget 16384 (compaction workload).
* ``q32b``   8 KV heads / 64 query heads, d=128, 131072 tokens, 64-token pages,
             128-row windows, budget 32768.
* ``stress`` the ``q8b`` layer with 30% of eligible pages forced to high-to-low
             (their keys aligned with the pre window x3 mass and the post
             window x0.2 mass), joint test over up to 256 candidates,
             compaction to 25% of the cache.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

ENTROPY = 2608_07855

REASONING, TOOL_CALL, OBSERVATION = 0, 1, 2

_CFG_INDEX = {"tiny": 0, "q8b": 1, "q8b_stack": 2, "q32b": 3, "stress": 4}


@dataclass(frozen=True)
class Workload:
    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_tokens: int
    page_size: int
    window: int
    event_lo: int
    event_hi: int
    obs_len: int
    heavy_frac: float
    budget: int
    eta: float = 0.125
    max_pending_pages: int = 16
    n_layers: int = 1
    n_seq: int = 1
    forced_frac: float = 0.0
    max_cand: int = 0          # 0: no cap
    gapped_positions: bool = False


WORKLOADS = {
    "tiny": Workload("tiny", 4, 1, 64, 2048, 16, 32, 32, 256, 128, 0.02, 1024),
    "q8b": Workload("q8b", 32, 8, 128, 32768, 32, 64, 64, 2048, 128, 0.01, 8192),
    "q8b_stack": Workload("q8b_stack", 32, 8, 128, 65536, 32, 64, 64, 2048, 128,
                          0.01, 16384, n_layers=36, n_seq=4),
    "q32b": Workload("q32b", 64, 8, 128, 131072, 64, 128, 64, 2048, 128, 0.01,
                     32768),
    "stress": Workload("stress", 32, 8, 128, 32768, 32, 64, 64, 2048, 128, 0.01,
                       8192, forced_frac=0.30, max_cand=256),
}


def scaled(base: str, **over) -> Workload:
    """A named workload with some fields replaced (for small parity cases)."""
    d = dict(WORKLOADS[base].__dict__)
    d.update(over)
    return Workload(**d)


def rng_for(w: Workload, seed: int, seq: int, layer: int, stream: int):
    ss = np.random.SeedSequence(
        entropy=ENTROPY + seed,
        spawn_key=(_CFG_INDEX.get(w.name, 99), seq, layer, stream))
    return np.random.Generator(np.random.PCG64(ss))


# stream ids
_S_LAYOUT, _S_K, _S_V, _S_HEAVY, _S_QPRE, _S_QPOST, _S_FORCED, _S_SCORE = range(8)


def bf16_bits(x_f32: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x_f32, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass
class Layout:
    """Event layout of one sequence (token index = position before gaps)."""
    n_tokens: int
    events: list                 # (kind, start, length)
    s_pre: int                   # cache prefix resident at the pre-commit window
    tool_call: tuple             # (start, length) of the committed tool call a_t
    observation: tuple           # (start, length) of its observation o_t
    page_start: np.ndarray       # pages of E_c (tool calls + observations in [0, s_pre))
    page_len: np.ndarray
    page_kind: np.ndarray
    pending_idx: np.ndarray      # indices (into the page list) of a_t's pages
    qrows_pre: np.ndarray        # token indices of the pre-commit window rows
    qrows_post: np.ndarray       # token indices of the post-commit window rows


def make_layout(w: Workload, rng) -> Layout:
    S, W = w.n_tokens, w.window
    la = max(int(rng.integers(w.event_lo, w.event_hi + 1)), W)
    head_end = S - W - w.obs_len - la
    if head_end < 0:
        raise ValueError("cache too short for the commit tail")
    events, t, kinds = [], 0, (REASONING, TOOL_CALL, OBSERVATION)
    k = 0
    while t < head_end:
        ln = int(rng.integers(w.event_lo, w.event_hi + 1))
        ln = min(ln, head_end - t)
        events.append((kinds[k % 3], t, ln))
        t += ln
        k += 1
    events.append((TOOL_CALL, head_end, la))
    events.append((OBSERVATION, head_end + la, w.obs_len))
    events.append((REASONING, head_end + la + w.obs_len, W))
    s_pre = head_end + la
    ps, pl, pk = [], [], []
    pending = []
    for kind, st, ln in events:
        if kind == REASONING or st + ln > s_pre:
            continue
        for off in range(0, ln, w.page_size):
            if st == head_end:
                pending.append(len(ps))
            ps.append(st + off)
            pl.append(min(w.page_size, ln - off))
            pk.append(kind)
    return Layout(S, events, s_pre, (head_end, la), (head_end + la, w.obs_len),
                  np.array(ps, np.int32), np.array(pl, np.int32),
                  np.array(pk, np.int8), np.array(pending, np.int64),
                  np.arange(s_pre - W, s_pre), np.arange(S - W, S))


@dataclass
class LayerInputs:
    w: Workload
    layout: Layout
    k: np.ndarray        # uint16 bf16 bits [Hkv, S, d]
    v: np.ndarray        # uint16 bf16 bits [Hkv, S, d]
    pos: np.ndarray      # int32 [S]
    q_pre: np.ndarray    # uint16 [Hq, W, d]
    q_post: np.ndarray   # uint16 [Hq, W, d]
    qpos_pre: np.ndarray   # int32 [W]
    qpos_post: np.ndarray  # int32 [W]
    forced: np.ndarray = field(default_factory=lambda: np.zeros(0, bool))

    @property
    def pages(self):
        return list(zip(self.layout.page_start.tolist(), self.layout.page_len.tolist()))


def _normal_bf16(rng, shape):
    return bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def make_layer(w: Workload, seed: int = 0, seq: int = 0, layer: int = 0) -> LayerInputs:
    """One layer of one sequence: bf16 N(0,1) K/V/Q, heavy-hitter keys x4."""
    lay = make_layout(w, rng_for(w, seed, seq, 0, _S_LAYOUT))
    S, d, Hkv, Hq, W = w.n_tokens, w.head_dim, w.n_kv_heads, w.n_q_heads, w.window
    k = _normal_bf16(rng_for(w, seed, seq, layer, _S_K), (Hkv, S, d))
    v = _normal_bf16(rng_for(w, seed, seq, layer, _S_V), (Hkv, S, d))
    n_heavy = int(round(w.heavy_frac * S))
    if n_heavy:
        heavy = rng_for(w, seed, seq, layer, _S_HEAVY).choice(S, n_heavy, replace=False)
        kf = bf16_bits_to_f32(k[:, heavy, :]) * np.float32(4.0)   # exact in bf16
        k[:, heavy, :] = bf16_bits(kf)
    q_pre = _normal_bf16(rng_for(w, seed, seq, layer, _S_QPRE), (Hq, W, d))
    q_post = _normal_bf16(rng_for(w, seed, seq, layer, _S_QPOST), (Hq, W, d))
    if w.gapped_positions:
        gaps = rng_for(w, seed, seq, 0, _S_LAYOUT + 100).integers(1, 4, S)
        pos = (np.cumsum(gaps) - gaps[0]).astype(np.int32)
    else:
        pos = np.arange(S, dtype=np.int32)
    forced = np.zeros(len(lay.page_start), bool)
    if w.forced_frac > 0:
        forced = _force_pages(w, lay, k, q_pre, q_post, seed, seq, layer)
    return LayerInputs(w, lay, k, v, pos, q_pre, q_post,
                       pos[lay.qrows_pre].astype(np.int32),
                       pos[lay.qrows_post].astype(np.int32), forced)


def _force_pages(w, lay, k, q_pre, q_post, seed, seq, layer):
    """Stress construction: a logit offset of +ln 3 in the pre window and
    ln 0.2 in the post window on the keys of 30% of the eligible pages.

    Key axis 0 is zeroed everywhere, set to kappa = sqrt(d) on forced tokens,
    and every query row gets axis 0 = ln(c) * sqrt(d) / kappa, so a forced
    token's logit moves by ln(c) (up to bf16 rounding) and no other logit moves.
    """
    n = len(lay.page_start)
    rng = rng_for(w, seed, seq, layer, _S_FORCED)
    n_forced = int(round(w.forced_frac * n))
    forced = np.zeros(n, bool)
    forced[rng.choice(n, n_forced, replace=False)] = True
    d = w.head_dim
    kappa = float(bf16_bits_to_f32(bf16_bits(np.array([math.sqrt(d)], np.float32)))[0])
    k[:, :, 0] = 0
    kap_bits = bf16_bits(np.array([kappa], np.float32))[0]
    for j in np.flatnonzero(forced):
        st, ln = int(lay.page_start[j]), int(lay.page_len[j])
        k[:, st:st + ln, 0] = kap_bits
    q_pre[:, :, 0] = bf16_bits(np.array([math.log(3.0) * math.sqrt(d) / kappa], np.float32))[0]
    q_post[:, :, 0] = bf16_bits(np.array([math.log(0.2) * math.sqrt(d) / kappa], np.float32))[0]
    return forced


def make_scores(n_tokens: int, seed: int = 0, ties: bool = False) -> np.ndarray:
    """A float32 score per token for selection-only tests (optionally with ties)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        entropy=ENTROPY + seed, spawn_key=(99, _S_SCORE))))
    s = rng.standard_normal(n_tokens).astype(np.float32)
    if ties:
        s = np.round(s * 4).astype(np.float32) / 4
    return s
