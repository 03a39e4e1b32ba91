"""Seeded synthetic multi-turn agent trajectories (no method arithmetic).

A trajectory stands in for one ReAct episode of the paper's agent benchmarks
(Sec. 3.1, Eq. (1); Sec. 4.1): a prompt, then turns of reasoning z_t, a tool
call a_t and the returned observation o_t, the last turn ending in an answer
instead of a tool call.  Every token is identified by its absolute position;
its keys, values and queries (every layer and head) are a pure function of
(trajectory, seed, sequence, layer, position), drawn chunk by chunk from
counter-keyed PCG64 streams, so any side can materialise any token range
without replaying the episode.

``schedule`` turns an episode into the order in which an engine would see it
(Algorithm 1 and the protocol of Sec. 4.1): prefilled events, decoded tokens,
the post-commit window of the previous commit once its first W reasoning
tokens exist, a compression checkpoint after every ``checkpoint_every``
decoded tokens, and the pre-commit measurement when a tool call ends.  It is
the caller's loop, not part of the method: both the oracle and the library's
lifecycle driver consume the same schedule.

Named trajectories:

* ``tiny_agent``  1 KV head / 4 query heads, d=64, 2 layers, 16-token pages,
                  16-row windows, budget 512, 6-8 turns.
* ``paper_agent`` the paper's operating point (Sec. 4.1): W=8, G=16,
                  eta=0.125, at most 64 scanned and 16 protected pages,
                  checkpoints every 128 decoded tokens, budget 4096, on a
                  Qwen3-14B-shaped layer stack (40 query / 8 KV heads, d=128).
* ``q8b_agent``   Qwen3-8B-shaped stack (32 / 8 heads, d=128, 36 layers),
                  32-token pages, 64-row windows, budget 16384, 20-60 turns.

With ``forced_frac`` > 0 a fraction of the tool-call and observation pages
is forced towards a high-to-low transition, as in the single-layer stress
workload: key axis 0 is zero except on forced tokens (kappa = sqrt(d)), and
query axis 0 is ln(forced_pre) sqrt(d) / kappa on tool-call tokens (so the
pre-commit window, the end of a tool call, gives forced tokens forced_pre
times their mass) and ln(forced_post) sqrt(d) / kappa on reasoning tokens
(the post-commit window).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np

from .workloads import ENTROPY, OBSERVATION, REASONING, TOOL_CALL, bf16_bits, bf16_bits_to_f32

PROMPT, ANSWER = 3, 4
DECODED_KINDS = (REASONING, TOOL_CALL, ANSWER)

_TRAJ_INDEX = {"tiny_agent": 10, "paper_agent": 11, "q8b_agent": 12}
_CHUNK = 512
_S_K, _S_V, _S_HEAVY, _S_Q, _S_TURNS, _S_FORCED = range(6)


@dataclass(frozen=True)
class TrajectoryConfig:
    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_layers: int
    page_size: int
    window: int
    prompt_lo: int
    prompt_hi: int
    reason_lo: int
    reason_hi: int
    call_lo: int
    call_hi: int
    obs_lo: int
    obs_hi: int
    turns_lo: int
    turns_hi: int
    budget: int
    eta: float = 0.125
    max_pending_pages: int = 16
    max_scan_pages: int = 64
    checkpoint_every: int = 128
    keep_recent: int = 0
    score_layer: int = 0
    heavy_frac: float = 0.01
    forced_frac: float = 0.0     # fraction of pages forced to a high-to-low transition
    forced_pre: float = 20.0     # attention-mass factor of tool-call queries on forced pages
    forced_post: float = 0.02    # ... of reasoning queries
    pool_kernel: int = 0         # base score pooled over this many tokens (0: not pooled)
    pool_mode: str = "max"

    @property
    def capacity(self) -> int:
        """Token slots a cache buffer needs: the budget, the tokens decoded
        between two checkpoints, the prompt, and every observation that can
        arrive between two checkpoints (a turn decodes at least 2 W tokens)."""
        per_turn = max(self.window, self.reason_lo) + max(self.window, self.call_lo)
        n_obs = self.checkpoint_every // per_turn + 1
        return self.budget + self.checkpoint_every + self.prompt_hi + n_obs * self.obs_hi + 64


TRAJECTORIES = {
    "tiny_agent": TrajectoryConfig("tiny_agent", 4, 1, 64, 2, 16, 16, 64, 128, 16, 96, 16, 64,
                                   32, 256, 6, 8, 512, keep_recent=16, score_layer=1,
                                   heavy_frac=0.005, forced_frac=0.15, forced_pre=100.0,
                                   forced_post=0.005),
    "paper_agent": TrajectoryConfig("paper_agent", 40, 8, 128, 40, 16, 8, 256, 1024, 64, 1024,
                                    16, 256, 64, 2048, 20, 60, 4096, keep_recent=8,
                                    score_layer=20),
    "q8b_agent": TrajectoryConfig("q8b_agent", 32, 8, 128, 36, 32, 64, 256, 1024, 64, 2048,
                                  64, 512, 64, 2048, 20, 60, 16384, keep_recent=64,
                                  score_layer=18),
}


def scaled_trajectory(base: str, **over) -> TrajectoryConfig:
    return replace(TRAJECTORIES[base], **over)


@dataclass
class Trajectory:
    cfg: TrajectoryConfig
    seed: int
    seq: int
    events: list        # (kind, start, length), absolute positions, in order
    forced: list = None  # forced pages (start, length)

    @property
    def n_tokens(self) -> int:
        kind, st, ln = self.events[-1]
        return st + ln


def _rng(cfg, seed, seq, layer, stream, chunk=0):
    ss = np.random.SeedSequence(entropy=ENTROPY + seed,
                                spawn_key=(_TRAJ_INDEX.get(cfg.name, 98), seq, layer, stream, chunk))
    return np.random.Generator(np.random.PCG64(ss))


def make_trajectory(cfg: TrajectoryConfig, seed: int = 0, seq: int = 0, n_turns: int | None = None) -> Trajectory:
    """Event lengths uniform in the configured ranges; reasoning and tool
    calls are at least W tokens long so both windows lie inside them."""
    r = _rng(cfg, seed, seq, 0, _S_TURNS)
    W = cfg.window
    T = n_turns if n_turns is not None else int(r.integers(cfg.turns_lo, cfg.turns_hi + 1))
    ev, p = [], 0

    def add(kind, n):
        nonlocal p
        ev.append((kind, p, int(n)))
        p += int(n)

    add(PROMPT, r.integers(cfg.prompt_lo, cfg.prompt_hi + 1))
    for t in range(1, T + 1):
        add(REASONING, max(W, int(r.integers(cfg.reason_lo, cfg.reason_hi + 1))))
        if t == T:
            add(ANSWER, max(W, int(r.integers(cfg.call_lo, cfg.call_hi + 1))))
            break
        add(TOOL_CALL, max(W, int(r.integers(cfg.call_lo, cfg.call_hi + 1))))
        add(OBSERVATION, r.integers(cfg.obs_lo, cfg.obs_hi + 1))
    forced = []
    if cfg.forced_frac > 0:
        fr = _rng(cfg, seed, seq, 0, _S_FORCED)
        for kind, st, ln in ev:
            if kind in (TOOL_CALL, OBSERVATION):
                for off in range(0, ln, cfg.page_size):
                    if fr.random() < cfg.forced_frac:
                        forced.append((st + off, min(cfg.page_size, ln - off)))
    return Trajectory(cfg, seed, seq, ev, forced)


def _kappa(cfg):
    return float(bf16_bits_to_f32(bf16_bits(np.array([math.sqrt(cfg.head_dim)], np.float32)))[0])


def _forced_mask(traj, p0, p1):
    m = np.zeros(max(p1 - p0, 0), bool)
    for st, ln in traj.forced or ():
        a, b = max(st, p0), min(st + ln, p1)
        if a < b:
            m[a - p0:b - p0] = True
    return m


def _kinds(traj, p0, p1):
    out = np.full(max(p1 - p0, 0), -1, np.int64)
    for kind, st, ln in traj.events:
        a, b = max(st, p0), min(st + ln, p1)
        if a < b:
            out[a - p0:b - p0] = kind
    return out


def _chunk_rows(cfg, traj, layer, stream, chunk, heads):
    r = _rng(cfg, traj.seed, traj.seq, layer, stream, chunk)
    x = bf16_bits(r.standard_normal((heads, _CHUNK, cfg.head_dim), dtype=np.float32))
    if stream == _S_K and cfg.heavy_frac > 0:
        hv = _rng(cfg, traj.seed, traj.seq, layer, _S_HEAVY, chunk).random(_CHUNK) < cfg.heavy_frac
        if hv.any():
            x[:, hv, :] = bf16_bits(bf16_bits_to_f32(x[:, hv, :]) * np.float32(4.0))   # exact in bf16
    return x


def _rows(cfg, traj, layer, stream, heads, p0, p1):
    out = np.empty((heads, max(p1 - p0, 0), cfg.head_dim), np.uint16)
    c = p0 // _CHUNK
    while c * _CHUNK < p1:
        a, b = max(p0, c * _CHUNK), min(p1, (c + 1) * _CHUNK)
        out[:, a - p0:b - p0] = _chunk_rows(cfg, traj, layer, stream, c, heads)[:, a - c * _CHUNK:b - c * _CHUNK]
        c += 1
    return out


def kv_rows(traj: Trajectory, layer: int, p0: int, p1: int):
    """bf16 bits of the keys and values at positions [p0, p1): [Hkv, n, d] each.
    Keys are N(0,1) with a fraction heavy_frac scaled by 4 (shared by the KV
    heads of a layer); values N(0,1)."""
    cfg = traj.cfg
    k = _rows(cfg, traj, layer, _S_K, cfg.n_kv_heads, p0, p1)
    if cfg.forced_frac > 0:
        k[:, :, 0] = 0
        k[:, _forced_mask(traj, p0, p1), 0] = bf16_bits(np.array([_kappa(cfg)], np.float32))[0]
    return k, _rows(cfg, traj, layer, _S_V, cfg.n_kv_heads, p0, p1)


def query_rows(traj: Trajectory, layer: int, p0: int, p1: int):
    """bf16 bits of the queries at positions [p0, p1): [Hq, n, d], N(0,1)."""
    cfg = traj.cfg
    q = _rows(cfg, traj, layer, _S_Q, cfg.n_q_heads, p0, p1)
    if cfg.forced_frac > 0:
        kinds = _kinds(traj, p0, p1)
        s = math.sqrt(cfg.head_dim) / _kappa(cfg)
        q[:, :, 0] = 0
        for kind, c in ((TOOL_CALL, cfg.forced_pre), (REASONING, cfg.forced_post)):
            q[:, kinds == kind, 0] = bf16_bits(np.array([math.log(c) * s], np.float32))[0]
    return q


def schedule(traj: Trajectory):
    """The engine's order of operations over the episode.

    Actions (positions absolute):
      ("append", kind, p0, p1, decoded, begins_event)  tokens [p0, p1) enter the cache
      ("post", p0)        post-commit window [p0, p0 + W) of the pending commit
      ("checkpoint", p0)  compression checkpoint; score window [p0, p0 + W)
      ("commit", p0)      commit at the end of a tool call; window [p0, p0 + W)

    A decoded event is split so that every action falls between two appends:
    the post window is complete after the first W tokens of the reasoning
    that follows an observation, and a checkpoint is due after every
    checkpoint_every decoded tokens (counted across events and turns).  When
    both fall on the same token the post measurement comes first.
    """
    cfg = traj.cfg
    W, C = cfg.window, cfg.checkpoint_every
    acts, decoded, commit_open, post_at = [], 0, False, None
    for kind, st, ln in traj.events:
        if kind not in DECODED_KINDS:
            acts.append(("append", kind, st, st + ln, False, True))
            continue
        if kind == REASONING and commit_open:
            post_at = st + W
        p = st
        while p < st + ln:
            stop = min(st + ln, p + (C - decoded % C))
            if post_at is not None and post_at > p:
                stop = min(stop, post_at)
            acts.append(("append", kind, p, stop, True, p == st))
            decoded += stop - p
            p = stop
            if post_at is not None and p == post_at:
                acts.append(("post", p - W))
                post_at, commit_open = None, False
            if decoded % C == 0:
                acts.append(("checkpoint", p - W))
        if kind == TOOL_CALL:
            acts.append(("commit", st + ln - W))
            commit_open = True
    return acts
