#!/usr/bin/env python3
"""Benchmark of the CommitKV hot path on one MI355X.

One step is one pass of the whole path over one commit of the synthetic
Qwen3-8B-shaped layer (32 query heads, 8 KV heads, head width 128, 32768
cached tokens, 32-token pages, 64-row windows, budget 8192):

  1. page deletion effects in the pre-commit window (cache prefix),
  2. page deletion effects in the post-commit window (full cache), with the
     window outputs and the token window-mass used as the base score,
  3. lifecycle classification and the ordered candidate list,
  4. the greedy joint test on the candidates,
  5. pending protection, budgeted selection and compaction of K, V and
     positions with one index set.

Inputs are resident in HBM before timing starts.  The key/value cache is
held in four copies and consecutive measurement calls read different copies,
so no call finds its keys and values still in the 256 MB Infinity Cache (a
real agent decodes many tokens over the whole cache between the two windows).

Prints one JSON line.  ``value`` = cached tokens scored per second per layer,
(S_pre + S_post) / step time.  Extra fields give the measurement-only rate,
the compaction bandwidth and per-kernel times (HIP events recorded by the
library on its stream).  ``roofline`` is for the kernel with the largest
total time; ``cpu_baseline`` times the fp64 oracle on a bounded sample on the
host cores.  ``recorded`` times the per-page pass alone from recorded window
outputs (ckv_measure_recorded); ``paged`` the measurement over a paged pool;
``stack`` the per-layer measurement of 36 layers x 4 sequences at 65536
tokens through the batched call.  ``agent`` runs whole synthetic agent episodes of a 36-layer stack
through the lifecycle driver (Algorithm 1) and reports the driver's time per
commit, post-commit step and checkpoint; ``agent_paper_point`` does the same
at the paper's operating point (W 8, G 16, budget 4096, 40 layers;
``agent_paper_budgets`` repeats it at budgets 2048 and 8192), and
``agent_paged`` runs the first workload's episodes with a paged agent (pool
rows in scattered order; a checkpoint re-indexes the slot table instead of
moving keys and values).  ``step_ms_events`` gives the median and 10th / 90th
percentiles of single steps timed with events; ``configs`` the pre + post
measurement alone on every synthetic workload (2K to 128K cached tokens, the
forced-page stress case included) with its roofline fraction.
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "cached tokens scored/sec per layer (pre+post commit) at 32K ctx; compaction GB/s"
PEAK_HBM = 8.0e12          # bytes/s
PEAK_MFMA = 2.5e15         # dense bf16/fp16 FLOP/s
RIDGE = PEAK_MFMA / PEAK_HBM


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="q8b")
    ap.add_argument("--copies", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-agent", action="store_true",
                    help="skip the lifecycle-driver leg (whole agent episodes, Algorithm 1)")
    ap.add_argument("--agent-seqs", type=int, default=4)
    ap.add_argument("--no-stack", action="store_true",
                    help="skip the 144-problem stack leg (36 layers x 4 sequences at 65536 tokens)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload pre + post measurement leg")
    ap.add_argument("--no-recorded", action="store_true",
                    help="skip the recorded-output leg (ckv_measure_recorded)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (5 launches), the known-size "
                         "reference that scales the FETCH_SIZE / WRITE_SIZE counters")
    return ap.parse_args()


def calibrate_copy(mib):
    """A plain copy of known size: under rocprofv3 --pmc its FETCH_SIZE and
    WRITE_SIZE per dispatch give the factor between the counters and bytes."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4, "launches": 5}), flush=True)


class Setup:
    def __init__(self, w, copies):
        import torch

        import paper_2608_07855_amd as P
        from synth import make_layer

        self.P, self.w = P, w
        t0 = time.time()
        L = make_layer(w, seed=0)
        self.L = L
        log(f"[bench] generated {w.name}: S={w.n_tokens} S_pre={L.layout.s_pre} pages={len(L.pages)} "
            f"({time.time() - t0:.1f}s)")

        def dev16(a):
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

        k0, v0 = dev16(L.k), dev16(L.v)
        self.k = [k0] + [k0.clone() for _ in range(copies - 1)]
        self.v = [v0] + [v0.clone() for _ in range(copies - 1)]
        self.pos = torch.from_numpy(L.pos).cuda()
        self.pos2 = self.pos[None]
        qpre, qpost = dev16(L.q_pre), dev16(L.q_post)
        qp_pre, qp_post = torch.from_numpy(L.qpos_pre).cuda(), torch.from_numpy(L.qpos_post).cuda()
        self.kv_pre = [P.kv_view(k, v, self.pos, L.layout.s_pre) for k, v in zip(self.k, self.v)]
        self.kv_post = [P.kv_view(k, v, self.pos) for k, v in zip(self.k, self.v)]
        self.win_pre = P.window_view(qpre, qp_pre)
        self.win_post = P.window_view(qpost, qp_post)
        self.pages = P.Pages(L.layout.page_start, L.layout.page_len)
        n = len(L.pages)
        self.n_pages = n
        pend = L.layout.pending_idx
        assert np.array_equal(pend, np.arange(pend[0], pend[-1] + 1))
        self.pend_slice = slice(int(pend[0]), int(pend[-1]) + 1)
        self.pending = P.Pages(L.layout.page_start[pend], L.layout.page_len[pend])
        self.force = torch.from_numpy(L.forced.astype(np.uint8)).cuda() if L.forced.any() else None
        self.max_cand = w.max_cand if w.max_cand > 0 else 256
        Hq, W, d, S = w.n_q_heads, w.window, w.head_dim, w.n_tokens
        f32 = dict(dtype=torch.float32, device="cuda")
        self.R_pre = torch.empty(n, **f32)
        self.R_post = torch.empty(n, **f32)
        self.o = torch.empty(Hq * W * d, **f32)
        self.lse = torch.empty(Hq * W, **f32)
        self.mass = torch.empty(S, **f32)
        B = w.budget
        self.k_out = torch.empty((1, 1, w.n_kv_heads, B, d), dtype=torch.bfloat16, device="cuda")
        self.v_out = torch.empty_like(self.k_out)
        self.pos_out = torch.empty((1, B), dtype=torch.int32, device="cuda")
        self.k5 = [k[None, None] for k in self.k]
        self.v5 = [v[None, None] for v in self.v]
        self.no_pages = P.Pages([], [])
        self.R_none = torch.empty(1, **f32)
        self.kept = torch.empty((1, B), dtype=torch.int32, device="cuda")
        self.n_kept = torch.empty(1, dtype=torch.int32, device="cuda")
        self.ctx = P.Context(0)
        self.last = {}

    def step(self, i, ev=None):
        """One pass of the whole path.  ``ev``: a pair of events recorded on
        the library's stream around the two measurement calls (the
        measurement pass of Sec. 3.2: window attention, per-page effects
        and their fix-up, R written)."""
        P, w = self.P, self.w
        c_pre, c_post = (2 * i) % len(self.k), (2 * i + 1) % len(self.k)
        if ev is not None:
            ev[0].record()
        P.ckv_measure_page_effects(self.ctx, self.kv_pre[c_pre], self.win_pre, self.pages, R=self.R_pre)
        P.ckv_measure_page_effects(self.ctx, self.kv_post[c_post], self.win_post, self.pages,
                                   R=self.R_post, o=self.o, lse=self.lse)
        if ev is not None:
            ev[1].record()
        # the base score of the selection: the post window's attention mass of
        # every token, from the window outputs just measured (no pages)
        P.ckv_measure_recorded(self.ctx, self.kv_post[c_post], self.win_post, self.no_pages, self.o, self.lse,
                               R=self.R_none, token_mass=self.mass)
        cl = P.ckv_classify_pages(self.ctx, self.R_pre, self.R_post, force=self.force,
                                  max_cand=self.max_cand)
        jt = P.ckv_joint_test(self.ctx, self.kv_post[c_post], self.win_post, self.o, self.lse,
                              self.pages, cl["cand"], cl["n_cand"], self.max_cand, 0.01)
        # the accepted pages join the retired set (Algorithm 1) on the device
        out = P.ckv_select_and_compact(
            self.ctx, self.k5[c_post], self.v5[c_post], self.pos2, [w.n_tokens], self.mass[None],
            [self.no_pages], [self.pending], [self.R_pre[self.pend_slice]], budget=w.budget, eta=w.eta,
            max_pending_pages=w.max_pending_pages, keep_recent=w.window,
            k_out=self.k_out, v_out=self.v_out, pos_out=self.pos_out,
            accepted=[(self.pages, cl["cand"], cl["n_cand"], jt["accepted"], self.max_cand)],
            kept=self.kept, n_kept=self.n_kept)
        self.last = dict(cl=cl, jt=jt, sel=out)


def recorded_leg(st, steps):
    """The per-page pass alone, from recorded window outputs
    (ckv_measure_recorded): the outputs and log-sum-exp of both windows are
    taken once (the engine records them in its forward pass), then each timed
    step runs the pre and post passes (the post one with the token mass)."""
    import torch
    P = st.P
    rec = []
    for kv, win in ((st.kv_pre[0], st.win_pre), (st.kv_post[0], st.win_post)):
        m = P.ckv_measure_page_effects(st.ctx, kv, win, st.pages, want=("R", "o", "lse"))
        rec.append((m["o"].contiguous(), m["lse"].contiguous()))
    n = len(st.k)

    def step(i):
        P.ckv_measure_recorded(st.ctx, st.kv_pre[(2 * i) % n], st.win_pre, st.pages, *rec[0], R=st.R_pre)
        P.ckv_measure_recorded(st.ctx, st.kv_post[(2 * i + 1) % n], st.win_post, st.pages, *rec[1],
                               R=st.R_post, token_mass=st.mass)

    for i in range(3):
        step(i)
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(i)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    gc.enable()
    toks = st.L.layout.s_pre + st.w.n_tokens
    return dict(ms_per_step=ms, tokens_per_s=toks / (ms / 1e3),
                note="pre + post page effects and token mass from recorded window outputs "
                     "(ckv_measure_recorded); no window-attention pass")


def paged_leg(st, steps):
    """The measurement passes (pre and post, with token mass) over a paged
    pool: the layer's tokens scattered over 1.5 S rows of each head's
    storage, addressed through a slot table (ckv_kv_view.slot)."""
    import torch
    P, L, w = st.P, st.L, st.w
    S = w.n_tokens
    rows = S + S // 2
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    slot = torch.randperm(rows, generator=g, device="cuda")[:S].to(torch.int32)
    kp = torch.zeros((w.n_kv_heads, rows, w.head_dim), dtype=torch.bfloat16, device="cuda")
    vp = torch.zeros_like(kp)
    kp[:, slot.long()] = st.k[0]
    vp[:, slot.long()] = st.v[0]
    kv_pre = P.kv_view(kp, vp, st.pos, n_tokens=L.layout.s_pre, slot=slot[:L.layout.s_pre].contiguous())
    kv_post = P.kv_view(kp, vp, st.pos, slot=slot)

    def step():
        P.ckv_measure_page_effects(st.ctx, kv_pre, st.win_pre, st.pages, R=st.R_pre)
        P.ckv_measure_page_effects(st.ctx, kv_post, st.win_post, st.pages, R=st.R_post, o=st.o, lse=st.lse,
                                   token_mass=st.mass)

    for _ in range(3):
        step()
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    gc.enable()
    toks = L.layout.s_pre + S
    return dict(ms_per_step=ms, tokens_per_s=toks / (ms / 1e3),
                note="pre + post measurement with token mass over a paged pool of 1.5 S rows "
                     "(slot table); one pool, so the key/value rows may be reused from the Infinity Cache")


def stack_leg(steps, comp_reps=3):
    """Per-layer scoring of the full Qwen3-8B-shaped stack: 36 layers x 4
    sequences at 65536 cached tokens (144 problems, 38.6 GB of keys and
    values), each step running the pre- and the post-commit measurement of
    every problem through the batched call (ckv_measure_page_effects_batch);
    then the batched checkpoint of the same stack: one
    ckv_select_and_compact call that selects each sequence's index set
    (budget 16384, its pending tool-call pages protected) and compacts the
    keys and values of all 36 layers x 8 KV heads and the positions with it
    (Eq. (4)), timed with events.  Event layouts and page tables come from
    the seeded generator; keys, values, queries and the base scores are
    drawn by torch on the device (timing only)."""
    import torch

    import paper_2608_07855_amd as P
    from synth import WORKLOADS, make_layout
    from synth.workloads import rng_for

    w = WORKLOADS["q8b_stack"]
    S, Hkv, Hq, d, W = w.n_tokens, w.n_kv_heads, w.n_q_heads, w.head_dim, w.window
    NS, NL = w.n_seq, w.n_layers
    g = torch.Generator(device="cuda")
    g.manual_seed(11)

    def bf16(shape):
        return torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16)

    ctx = P.Context(0)
    # the whole stack in one tensor per K and V: [seq, layer, head, token, d]
    k5 = torch.empty((NS, NL, Hkv, S, d), dtype=torch.bfloat16, device="cuda")
    v5 = torch.empty_like(k5)
    pos2 = torch.arange(S, dtype=torch.int32, device="cuda")[None].repeat(NS, 1).contiguous()
    kv_pre, kv_post, w_pre, w_post, pages, keep, lays = [], [], [], [], [], [], []
    tokens = 0
    for sq in range(NS):
        lay = make_layout(w, rng_for(w, 0, sq, 0, 0))
        lays.append(lay)
        qp_pre = torch.from_numpy(lay.qrows_pre.astype(np.int32)).cuda()
        qp_post = torch.from_numpy(lay.qrows_post.astype(np.int32)).cuda()
        pg = P.Pages(lay.page_start, lay.page_len)
        for li in range(NL):
            k5[sq, li].copy_(bf16((Hkv, S, d)))
            v5[sq, li].copy_(bf16((Hkv, S, d)))
            q1, q2 = bf16((Hq, W, d)), bf16((Hq, W, d))
            keep += [q1, q2, qp_pre, qp_post]
            kv_pre.append(P.kv_view(k5[sq, li], v5[sq, li], pos2[sq], n_tokens=lay.s_pre))
            kv_post.append(P.kv_view(k5[sq, li], v5[sq, li], pos2[sq]))
            w_pre.append(P.window_view(q1, qp_pre))
            w_post.append(P.window_view(q2, qp_post))
            pages.append(pg)
            tokens += lay.s_pre + S
    n = len(kv_pre)
    R = [torch.empty(max(p.n, 1), dtype=torch.float32, device="cuda") for p in pages]

    def step():
        P.ckv_measure_page_effects_batch(ctx, kv_pre, w_pre, pages, R=R)
        P.ckv_measure_page_effects_batch(ctx, kv_post, w_post, pages, R=R)

    step()
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    gc.enable()
    out = dict(workload=f"qwen3-8b-shaped stack: {NL} layers x {NS} sequences at {S} cached tokens "
                        f"({n} problems), pre + post measurement per layer", problems=n,
               ms_per_step=ms, tokens_per_s=tokens / (ms / 1e3), tokens_per_step=tokens)
    # the batched checkpoint of the whole stack
    B = w.budget
    score = torch.rand((NS, S), generator=g, device="cuda")
    pend = [P.Pages(lay.page_start[lay.pending_idx], lay.page_len[lay.pending_idx]) for lay in lays]
    rpre = [torch.rand(max(p.n, 1), generator=g, device="cuda")[:p.n] for p in pend]
    no_pages = P.Pages([], [])
    k_out = torch.empty((NS, NL, Hkv, B, d), dtype=torch.bfloat16, device="cuda")
    v_out = torch.empty_like(k_out)
    pos_out = torch.empty((NS, B), dtype=torch.int32, device="cuda")
    kept = torch.empty((NS, B), dtype=torch.int32, device="cuda")
    n_kept = torch.empty(NS, dtype=torch.int32, device="cuda")

    def compact(_i):
        P.ckv_select_and_compact(ctx, k5, v5, pos2, [S] * NS, score, [no_pages] * NS, pend, rpre, budget=B,
                                 eta=w.eta, max_pending_pages=w.max_pending_pages, keep_recent=W,
                                 k_out=k_out, v_out=v_out, pos_out=pos_out, kept=kept, n_kept=n_kept)

    compact(0)
    cms = event_times(compact, comp_reps)
    nk = int(n_kept.sum().item())
    cbytes = 2 * nk * NL * Hkv * d * 2 * 2 + 2 * nk * 4
    q = pct(cms)
    out["checkpoint"] = dict(
        note=f"one ckv_select_and_compact call over {NS} sequences x {NL} layers x {Hkv} KV heads: per-sequence "
             f"selection of {B} of {S} tokens, then keys, values and positions gathered with one index set "
             "per sequence (Eq. (4)); bytes = read + write of the kept rows of every layer and head",
        kept_tokens=nk, bytes=cbytes, ms=q, GBps=cbytes / (q["median"] / 1e3) / 1e9,
        hbm_frac=cbytes / (q["median"] / 1e3) / PEAK_HBM)
    log(f"[bench] stack checkpoint: {q['median']:.3f} ms for {cbytes / 1e9:.2f} GB")
    ctx.close()
    del keep, k5, v5, k_out, v_out
    torch.cuda.empty_cache()
    return out


def joint_rounds(acc, window=32):
    """Rounds of the speculative joint test given its decisions: a round
    tests the next `window` candidates and ends at the first accepted one."""
    cur, rounds, n = 0, 0, len(acc)
    while cur < n:
        hit = next((t for t in range(cur, min(cur + window, n)) if acc[t]), None)
        cur = hit + 1 if hit is not None else cur + window
        rounds += 1
    return rounds


def stress_leg(reps=10):
    """The joint-test stress workload (Sec. 3.3, Eq. (11); Algorithm 1): the
    Qwen3-8B-shaped layer at 32768 tokens with 30% of its pages forced to
    high-to-low, those pages fed to the joint test as candidates in
    (R+ ascending, R- descending, start ascending) order, capped at 256, then
    the checkpoint that retires the accepted pages and compacts the cache to
    25% (budget 8192).  Joint test and checkpoint are timed with events,
    repeated on the same inputs."""
    import torch
    from synth import WORKLOADS

    w = WORKLOADS["stress"]
    st = Setup(w, 1)
    P, ctx = st.P, st.ctx
    P.ckv_measure_page_effects(ctx, st.kv_pre[0], st.win_pre, st.pages, R=st.R_pre)
    P.ckv_measure_page_effects(ctx, st.kv_post[0], st.win_post, st.pages, R=st.R_post, o=st.o, lse=st.lse)
    P.ckv_measure_recorded(ctx, st.kv_post[0], st.win_post, st.no_pages, st.o, st.lse, R=st.R_none,
                           token_mass=st.mass)
    own = P.ckv_classify_pages(ctx, st.R_pre, st.R_post)
    cl = P.ckv_classify_pages(ctx, st.R_pre, st.R_post, force=st.force, max_cand=st.max_cand)
    res = {}

    def joint(_i):
        res["jt"] = P.ckv_joint_test(ctx, st.kv_post[0], st.win_post, st.o, st.lse, st.pages, cl["cand"],
                                     cl["n_cand"], st.max_cand, 0.01)

    joint(0)
    jms = event_times(joint, reps)
    nc = int(cl["n_cand"].item())
    acc = res["jt"]["accepted"].cpu().numpy()[:nc]

    def checkpoint(_i):
        res["sel"] = P.ckv_select_and_compact(
            ctx, st.k5[0], st.v5[0], st.pos2, [w.n_tokens], st.mass[None], [st.no_pages], [st.pending],
            [st.R_pre[st.pend_slice]], budget=w.budget, eta=w.eta, max_pending_pages=w.max_pending_pages,
            keep_recent=w.window, k_out=st.k_out, v_out=st.v_out, pos_out=st.pos_out,
            accepted=[(st.pages, cl["cand"], cl["n_cand"], res["jt"]["accepted"], st.max_cand)],
            kept=st.kept, n_kept=st.n_kept)

    checkpoint(0)
    cms = event_times(checkpoint, reps)
    nk = int(st.n_kept[0].item())
    cbytes = 2 * nk * w.n_kv_heads * w.head_dim * 2 * 2 + 2 * nk * 4
    jq, cq = pct(jms), pct(cms)
    log(f"[bench] stress: joint {jq['median']:.3f} ms over {nc} candidates ({int(acc.sum())} accepted), "
        f"checkpoint {cq['median']:.3f} ms")
    out = dict(workload="qwen3-8b-shaped layer, 32768 tokens, 30% of pages forced high-to-low; candidates = the "
                        "forced pages in (R+ asc, R- desc, start asc) order, capped at 256; budget 8192 (25%)",
               classifier_candidates=int(own["n_cand"].item()), candidates=nc, accepted=int(acc.sum()),
               rounds=joint_rounds(acc), joint_ms=jq,
               checkpoint_ms=cq, kept_tokens=nk, checkpoint_bytes=cbytes,
               checkpoint_GBps=cbytes / (cq["median"] / 1e3) / 1e9)
    ctx.close()
    del st
    gc.collect()
    torch.cuda.empty_cache()
    return out


def agent_leg(n_seq, traj="q8b_agent", shape="qwen3-8b-shaped", paged=False, budget=None):
    """Whole agent episodes through the lifecycle driver (ckv_agent_*), one
    driver per episode: by default the Qwen3-8B-shaped stack (36 layers, 32
    query / 8 KV heads, d 128), budget 16384, 64-row windows, 32-token pages;
    ``paper_agent`` is the paper's operating point on a Qwen3-14B-shaped
    stack (40 layers, 40 / 8 heads, W 8, G 16, budget 4096); a checkpoint
    every 128 decoded tokens in both.  The engine's part (writing each new
    token's keys and values, drawing window queries) is synthetic torch work
    outside the timed calls; every commit, post and checkpoint is timed on
    the host around the call (each returns after the context's stream has
    finished it).  ``paged``: the agent scores one layer's pool through its
    slot table, and a checkpoint selects and re-indexes the table (the
    engine's per-layer pools stay where they are)."""
    import torch

    import paper_2608_07855_amd as P
    from synth.trajectory import TRAJECTORIES, make_trajectory, scaled_trajectory, schedule

    cfg = TRAJECTORIES[traj] if budget is None else scaled_trajectory(traj, budget=budget)
    ctx = P.Context(0)
    L, Hkv, d, Hq, W = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, cfg.n_q_heads, cfg.window
    t = dict(commit=0.0, post=0.0, checkpoint=0.0)
    n = dict(commit=0, post=0, checkpoint=0, compacted=0)
    moved, turns, tokens = 0, [], 0
    # a paged agent holds only the scoring layer's pool: the other layers'
    # pools are the engine's and the driver never touches them
    L_alloc = 1 if paged else L
    for s in range(n_seq):
        traj = make_trajectory(cfg, seed=0, seq=s)
        turns.append(sum(1 for e in traj.events if e[0] == 0))
        tokens += traj.n_tokens
        extra = dict(paged=True, pool_rows=cfg.capacity + 4096, row_seed=s) if paged else {}
        ag = P.Agent(ctx, L_alloc, Hkv, d, cfg.capacity, page_size=cfg.page_size, window=W, n_q_heads=Hq,
                     budget=cfg.budget, eta=cfg.eta, max_pending_pages=cfg.max_pending_pages,
                     keep_recent=cfg.keep_recent, max_scan_pages=cfg.max_scan_pages,
                     checkpoint_every=cfg.checkpoint_every, score_layer=0 if paged else cfg.score_layer,
                     **extra)
        g = torch.Generator(device="cuda")
        g.manual_seed(1000 + s)
        for act in schedule(traj):
            if act[0] == "append":
                _, kind, p0, p1, dec, first = act
                k = torch.randn((L_alloc, Hkv, p1 - p0, d), generator=g, device="cuda").to(torch.bfloat16)
                v = torch.randn((L_alloc, Hkv, p1 - p0, d), generator=g, device="cuda").to(torch.bfloat16)
                ag.append(kind, k, v, np.arange(p0, p1), dec, first)
                continue
            q = torch.randn((Hq, W, d), generator=g, device="cuda").to(torch.bfloat16)
            qp = torch.arange(act[1], act[1] + W, dtype=torch.int32, device="cuda")
            torch.cuda.synchronize()
            gc.disable()
            t0 = time.perf_counter()
            r = getattr(ag, act[0])(q, qp)
            t[act[0]] += time.perf_counter() - t0
            gc.enable()
            n[act[0]] += 1
            if act[0] == "checkpoint" and r["compacted"]:
                n["compacted"] += 1
                if not paged:
                    moved += len(r["kept"]) * (L * Hkv * d * 2 * 2 * 2 + 4 * 2)
        ag.close()
    ctx.close()
    total = sum(t.values())
    kv_b = cfg.budget * Hkv * d * 2 * 2
    log(f"[bench] agent leg: {n_seq} episodes, {tokens} tokens, driver time {total:.3f}s")
    return dict(
        workload=f"{shape} stack, {L} layers (Hq {Hq}, Hkv {Hkv}, d {d}), {n_seq} agent episodes "
                 f"of {cfg.turns_lo}-{cfg.turns_hi} turns, budget {cfg.budget}, {W}-row windows, "
                 f"{cfg.page_size}-token pages, a checkpoint every {cfg.checkpoint_every} decoded tokens"
                 + (", paged agent (pool rows in scattered order)" if paged else ""),
        turns=turns, tokens=tokens, driver_seconds=total, tokens_per_s=tokens / total if total else None,
        commits=n["commit"], posts=n["post"], checkpoints=n["checkpoint"], compactions=n["compacted"],
        ms_per_commit=1e3 * t["commit"] / max(n["commit"], 1), ms_per_post=1e3 * t["post"] / max(n["post"], 1),
        ms_per_checkpoint=1e3 * t["checkpoint"] / max(n["checkpoint"], 1),
        # one read of the scored layer's keys and values at the budget, at
        # 8 TB/s, against the host-timed call (commit: pre measurement; post:
        # post measurement, classification and joint test)
        layer_kv_bytes_at_budget=kv_b, kv_roofline_us=1e6 * kv_b / 8e12,
        commit_kv_roofline_frac=(kv_b / 8e12) / (t["commit"] / n["commit"]) if n["commit"] else None,
        post_kv_roofline_frac=(kv_b / 8e12) / (t["post"] / n["post"]) if n["post"] else None,
        compaction_GBps=moved / t["checkpoint"] / 1e9 if t["checkpoint"] > 0 and not paged else None)


def pct(ms):
    """median and 10th / 90th percentiles of a list of times"""
    a = np.asarray(ms, dtype=np.float64)
    return dict(median=float(np.median(a)), p10=float(np.percentile(a, 10)), p90=float(np.percentile(a, 90)))


def event_times(fn, reps):
    """fn(i) for i < reps, each bracketed by events on the current stream
    (the library's stream); per-call milliseconds"""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(ev):
        a.record()
        fn(i)
        b.record()
    torch.cuda.synchronize()
    gc.enable()
    return [a.elapsed_time(b) for a, b in ev]


def configs_leg(names=("tiny", "q8b", "q32b", "stress"), reps=30):
    """Cached tokens scored per second per layer on each synthetic workload:
    the pre and post measurement calls (R written; no token mass,
    classification or selection), each repetition bracketed by events, with
    the K/V copies rotated so that no call finds its cache in the 256 MB
    Infinity Cache.  ``roof_frac`` = t_roof / t_median with t_roof =
    max(bytes / 8 TB/s, FLOPs / 2.5 PFLOP/s) for one read of the resident
    keys, values and positions of both passes and the two products
    (Q K^T, P V) over them."""
    import torch
    from synth import WORKLOADS

    out = {}
    for name in names:
        w = WORKLOADS[name]
        st = Setup(w, 2 if w.n_tokens > 65536 else 4)
        P, n = st.P, len(st.k)

        def run(i):
            P.ckv_measure_page_effects(st.ctx, st.kv_pre[(2 * i) % n], st.win_pre, st.pages, R=st.R_pre)
            P.ckv_measure_page_effects(st.ctx, st.kv_post[(2 * i + 1) % n], st.win_post, st.pages, R=st.R_post)

        for i in range(5):
            run(i)
        ms = event_times(run, reps)
        toks = int(st.L.layout.s_pre) + w.n_tokens
        byt = toks * (w.n_kv_heads * w.head_dim * 2 * 2 + 4)
        flop = 4.0 * w.n_q_heads * w.window * toks * w.head_dim
        t_roof = max(byt / 8.0e12, flop / 2.5e15) * 1e3
        q = pct(ms)
        out[name] = dict(n_tokens=w.n_tokens, s_pre=int(st.L.layout.s_pre), pages=st.n_pages,
                         shape=f"Hq {w.n_q_heads} Hkv {w.n_kv_heads} d {w.head_dim} W {w.window} "
                               f"G {w.page_size}",
                         ms=q, tokens_per_s=toks / (q["median"] / 1e3), roof_ms=t_roof,
                         roof_frac=t_roof / q["median"])
        log(f"[bench] config {name}: median {q['median']:.3f} ms for pre + post")
        st.ctx.close()
        del st, run
        gc.collect()
        torch.cuda.empty_cache()
    return out


def pass_work(w, L):
    """Algorithmic bytes and FLOPs of the measurement pass pair (pre + post,
    Sec. 3.2): one read of each pass's resident keys, values and positions,
    the window queries, the outputs o and log-sum-exp, and R; FLOPs of the
    two products (Q K^T, P V) over the resident tokens."""
    Hq, Hkv, W, d, S, Sp = w.n_q_heads, w.n_kv_heads, w.window, w.head_dim, w.n_tokens, L.layout.s_pre
    rows = Hq * W
    toks = Sp + S
    byt = toks * (Hkv * d * 2 * 2 + 4) + 2 * (rows * d * 2 + rows * (d + 1) * 4 + len(L.pages) * 4)
    flop = 4.0 * rows * toks * d
    return byt, flop


def kernel_work(w, L, name, launches_per_step):
    """Algorithmic bytes and FLOPs per launch of a library kernel, and a note.
    The per-page pass (page_effect) re-reads the eligible keys and values
    that the window pass already read: that re-read is implementation
    traffic, not algorithmic, so its algorithmic bytes are only its own
    inputs and outputs (queries, o, R) and its fraction that matters is the
    MFMA one."""
    Hq, Hkv, W, d, S, Sp = w.n_q_heads, w.n_kv_heads, w.window, w.head_dim, w.n_tokens, L.layout.s_pre
    rows = Hq * W
    n_elig = int(L.layout.page_len.sum())
    note = None
    if name == "window_attention":      # one launch per pass: pre over S_pre, post over S
        toks = (Sp + S) / 2
        byt = toks * (Hkv * d * 2 * 2 + 4) + rows * d * 2 + rows * (d + 1) * 4
        flop = 4.0 * rows * toks * d
    elif name == "page_effect":         # eligible tokens, twice per step
        byt = rows * d * (2 + 4) + len(L.pages) * 4
        flop = 4.0 * rows * n_elig * d
        note = (f"re-reads the {n_elig} eligible tokens' keys and values "
                f"({n_elig * (Hkv * d * 2 * 2 + 4) / 1e6:.1f} MB per launch) after the window pass: "
                "implementation traffic, not counted as algorithmic")
    elif name in ("token_mass", "token_mass_fixup"):   # the latter also carries the post pass's fix-up
        byt = S * (Hkv * d * 2 + 4 + 4) + rows * d * 2
        flop = 2.0 * rows * S * d
    elif name == "gather":
        B = w.budget
        byt = B * Hkv * d * 2 * 2 * 2 + B * 4 * 3
        flop = 0.0
    else:
        return None
    return byt, flop, note


PASS_KERNELS = ("window_attention", "combine", "page_effect", "page_fixup")


def pass_traffic(workload):
    """HBM bytes (read + written) of one pre + post measurement pass pair
    from the committed counter summaries of its kernels (each scaled per
    step), or None if any of them is missing or its source has changed."""
    tot = 0.0
    for k in PASS_KERNELS:
        p = os.path.join(ROOT, "profiles", f"traffic_{k}_{workload}.json")
        if not os.path.exists(p):
            return None
        try:
            rec = json.load(open(p))
            if source_sha(os.path.join(ROOT, rec["source"])) != rec["source_sha256"]:
                return None
            tot += float(rec["bytes_per_launch"]) * float(rec.get("launches_per_step", 2))
        except Exception:
            return None
    return tot


def source_sha(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_for(kernel, workload):
    """HBM bytes per launch from committed rocprofv3 counter summaries, if they
    still match the kernel source; else None."""
    p = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(p):
        return None
    try:
        rec = json.load(open(p))
        src = os.path.join(ROOT, rec["source"])
        if source_sha(src) != rec["source_sha256"]:
            return None
        return float(rec["bytes_per_launch"])
    except Exception:
        return None


def cpu_baseline(w, L, budget_s):
    """Closed-form fp64 oracle (pre + post pass) on a sample of query heads,
    scaled to all heads; returns tokens per second."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_limits
    except Exception:
        threadpool_limits = None
    cores = len(os.sched_getaffinity(0))
    ctx = threadpool_limits(cores) if threadpool_limits else None
    Sp, S, Hq = L.layout.s_pre, w.n_tokens, w.n_q_heads
    heads, spent = [], 0.0
    t_all = time.time()
    for h in range(Hq):
        t0 = time.time()
        O.page_effects(L.k[:, :Sp], L.v[:, :Sp], L.pos[:Sp], L.q_pre, L.qpos_pre, L.pages,
                       method="closed", heads=[h])
        O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, method="closed", heads=[h])
        spent += time.time() - t0
        heads.append(h)
        if spent > budget_s:
            break
    if ctx is not None:
        ctx.unregister() if hasattr(ctx, "unregister") else None
    per_step = spent * Hq / len(heads)
    log(f"[bench] cpu oracle: {len(heads)} of {Hq} query heads in {spent:.1f}s "
        f"(wall {time.time() - t_all:.1f}s) -> {per_step:.1f}s per full pre+post pass")
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    return dict(value=(Sp + S) / per_step, unit="tokens/s", cores=cores, kind="oracle", cpu_model=model,
                sample=f"closed-form fp64 oracle, pre+post deletion effects of all {len(L.pages)} pages "
                       f"for query heads 0..{len(heads) - 1} of {Hq}, time scaled by {Hq}/{len(heads)}")


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}), flush=True)
        log("[bench] this build measures one GPU; multi-GPU runs are not part of it")
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    import torch
    from synth import WORKLOADS

    w = WORKLOADS[args.workload]
    st = Setup(w, args.copies)
    ctx = st.ctx
    for i in range(args.warmup):
        st.step(i)
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({args.warmup} steps)")
    # per-kernel breakdown: every kernel bracketed by events (this perturbs
    # the step, so it is measured on steps of its own)
    n_prof = max(args.steps // 2, 5)
    ctx.reset_kernel_stats()
    ctx.set_kernel_timing(True)
    for i in range(n_prof):
        st.step(args.warmup + i)
    ctx.set_kernel_timing(False)
    stats = ctx.kernel_stats()
    per_kernel = {k: dict(ms_per_step=v[0] / n_prof, launches_per_step=v[1] / n_prof)
                  for k, v in stats.items()}
    dom = max(per_kernel, key=lambda k: per_kernel[k]["ms_per_step"])
    # timed steps: events on the library's stream around each step's two
    # measurement calls (the pass roofline) and around the dominant kernel
    ctx.reset_kernel_stats()
    ctx.set_kernel_timing_only(dom)
    ctx.set_kernel_timing(True)
    pass_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
    # a full collection of the interpreter's objects stalls the host for tens
    # of milliseconds: collect now, none inside the timed steps
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        st.step(args.warmup + n_prof + i, pass_ev[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    gc.enable()
    ctx.set_kernel_timing(False)
    ctx.set_kernel_timing_only(None)
    dstats = ctx.kernel_stats()
    pass_ms = [a.elapsed_time(b) for a, b in pass_ev]
    ms = (t1 - t0) * 1e3 / args.steps
    L = st.L
    tokens = L.layout.s_pre + w.n_tokens
    value = tokens / (ms / 1e3)
    log(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step, measurement pass {np.mean(pass_ms):.3f} ms")
    # distribution of single steps (events around each), after the timed run
    step_dist = pct(event_times(lambda i: st.step(10_000 + i), max(args.steps, 30)))
    meas = sum(per_kernel.get(k, {}).get("ms_per_step", 0.0)
               for k in ("window_attention", "combine", "page_effect", "page_fixup"))
    sel_ms = sum(per_kernel.get(k, {}).get("ms_per_step", 0.0) for k in ("protect", "select", "gather"))
    g_ms = per_kernel.get("gather", {}).get("ms_per_step", 0.0)
    n_kept = int(st.last["sel"]["n_kept"][0].item())
    comp_bytes = 2 * n_kept * w.n_layers * w.n_kv_heads * w.head_dim * 2 * 2 + n_kept * 4 * 2
    # headline roofline: the measurement pass (pre + post), algorithmic bytes
    # = one read of each pass's resident keys, values and positions plus the
    # queries and the outputs, over the pass time from the events above
    pbyt, pflop = pass_work(w, L)
    pass_s = float(np.mean(pass_ms)) / 1e3
    roof = dict(bound="hbm", kernel="measurement pass (pre + post: window_attention, combine, page_effect, "
                                      "page_fixup)",
                achieved=pbyt / pass_s / 1e9, peak=PEAK_HBM / 1e9, unit="GB/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = pass_traffic(w.name)
    roof["algorithmic_bytes"] = pbyt
    roof["algorithmic_flop"] = pflop
    roof["mfma_frac"] = pflop / pass_s / PEAK_MFMA
    roof["pass_ms"] = pct(pass_ms)
    roof["roofline_ms"] = max(pbyt / PEAK_HBM, pflop / PEAK_MFMA) * 1e3
    # every library kernel of the step against its own bound
    kroof = {}
    for k in per_kernel:
        wk = kernel_work(w, L, k, per_kernel[k]["launches_per_step"])
        if not wk:
            continue
        byt, flop, note = wk
        avg_s = per_kernel[k]["ms_per_step"] / per_kernel[k]["launches_per_step"] / 1e3
        if k == dom and dom in dstats:
            avg_s = dstats[dom][0] / dstats[dom][1] / 1e3
        e = dict(avg_launch_us=avg_s * 1e6, algorithmic_bytes_per_launch=byt, flop_per_launch=flop,
                 hbm_frac=byt / avg_s / PEAK_HBM, mfma_frac=flop / avg_s / PEAK_MFMA,
                 traffic_bytes_per_launch=traffic_for(k, w.name))
        if note:
            e["note"] = note
        kroof[k] = e
    recorded = None if args.no_recorded else recorded_leg(st, args.steps)
    paged = None if args.no_recorded else paged_leg(st, args.steps)
    stack = None if args.no_stack else stack_leg(3)
    agent = None if args.no_agent else agent_leg(args.agent_seqs)
    agent_paper = None if args.no_agent else agent_leg(2, "paper_agent", "qwen3-14b-shaped, paper operating point")
    # the paper's other budgets (Sec. 4.1: B in {2048, 4096, 8192})
    agent_paper_budgets = None if args.no_agent else {
        str(b): agent_leg(2, "paper_agent", "qwen3-14b-shaped, paper operating point", budget=b)
        for b in (2048, 8192)}
    agent_paged = None if args.no_agent else agent_leg(args.agent_seqs, paged=True)
    configs = None if args.no_configs else configs_leg()
    stress = None if args.no_configs else stress_leg()
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, L, args.cpu_seconds)
    res = dict(
        metric=METRIC, value=value, unit="tokens/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
        ms_per_step=ms, step_ms_events=step_dist, higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="bf16",
        data="synthetic",
        config=dict(workload="qwen3-8b-shaped layer, 32768 cached tokens (Hq 32, Hkv 8, d 128, "
                             "32-token pages, 64-row windows, budget 8192)" if w.name == "q8b" else w.name,
                    name=w.name, n_tokens=w.n_tokens, s_pre=int(L.layout.s_pre), pages=len(L.pages),
                    parallelism="single GPU"),
        measure_only_tokens_per_s=tokens / pass_s,
        measure_kernels_tokens_per_s=tokens / (meas / 1e3) if meas > 0 else None,
        compaction_GBps=comp_bytes / (sel_ms / 1e3) / 1e9 if sel_ms > 0 else None,
        gather_GBps=comp_bytes / (g_ms / 1e3) / 1e9 if g_ms > 0 else None,
        compaction_note="the step compacts the copy the post pass has just streamed, so its kept rows may "
                        "still be in the 256 MB Infinity Cache; the stack leg's checkpoint (19.3 GB in one "
                        "call) is the figure no cache can hold",
        kernels=per_kernel,
        kernels_note="per-kernel times from separate profiling steps with events around every kernel",
        n_candidates=int(st.last["cl"]["n_cand"].item()),
        n_accepted=int(st.last["jt"]["n_accepted"].item()),
        n_kept=n_kept,
        roofline=roof,
        kernel_rooflines=kroof,
        cpu_baseline=cpu,
        recorded=recorded,
        paged=paged,
        stack=stack,
        agent=agent,
        agent_paper_point=agent_paper,
        agent_paper_budgets=agent_paper_budgets,
        agent_paged=agent_paged,
        configs=configs,
        stress=stress,
    )
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
