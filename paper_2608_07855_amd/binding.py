"""Thin Python binding of the CommitKV C ABI (include/commitkv.h).

Argument marshalling only: torch tensors supply device pointers, strides and
the current HIP stream; NumPy arrays supply the host page lists.  Every step
of the hot path runs in the HIP kernels of libcommitkv.so; there is no other
code path.  Each ``ckv_*`` function mirrors the C entry point of the same
name and returns the output tensors (allocating those the caller omits).
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np
import torch

from . import _abi
from ._abi import AcceptedPages, Budget, CacheView, KVView, PageList, Thresholds, WindowView

PAPER_THRESHOLDS = dict(tau_use=0.05, tau_dead=0.01, rho_use=0.75, rho_dead=0.25, tau_joint=0.01)


class CKVError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{_abi.STATUS_NAMES.get(code, code)}: {message}")
        self.code = code


def lib():
    return _abi.load()


def version() -> int:
    return int(lib().ckv_version())


class Context:
    """A ckv_ctx bound to one device and one HIP stream (default: torch's current)."""

    def __init__(self, device: int = 0, stream=None):
        self._lib = lib()
        if stream is None:
            stream = torch.cuda.current_stream(device).cuda_stream
        elif isinstance(stream, torch.cuda.Stream):
            stream = stream.cuda_stream
        self.device = device
        h = ctypes.c_void_p()
        rc = self._lib.ckv_create(ctypes.byref(h), device, ctypes.c_void_p(stream))
        if rc != 0:
            raise CKVError(rc, "ckv_create failed")
        self.handle = h

    def check(self, rc: int):
        if rc != 0:
            msg = self._lib.ckv_last_error(self.handle)
            raise CKVError(rc, msg.decode() if msg else "")

    def sync(self):
        self.check(self._lib.ckv_sync(self.handle))

    def set_stream(self, stream):
        s = stream.cuda_stream if isinstance(stream, torch.cuda.Stream) else stream
        self.check(self._lib.ckv_set_stream(self.handle, ctypes.c_void_p(s)))

    def set_workspace_limit(self, nbytes: int):
        self.check(self._lib.ckv_set_workspace_limit(self.handle, nbytes))

    def workspace_bytes(self) -> int:
        return int(self._lib.ckv_workspace_bytes(self.handle))

    def set_policy(self, *names):
        """Switch components off for the Sec. 4.4 ablation variants: names from
        no_precommit, no_percentile, no_joint, no_protection, no_lifecycle
        (none: the complete method)."""
        bits = 0
        for n in names:
            bits |= _abi.POLICY_BITS[n]
        self.check(self._lib.ckv_set_policy(self.handle, bits))

    def set_barrier_timeout_us(self, us: int):
        """Bound of a grid-wide wait in the joint test and the grid
        selection (0: give up unless every workgroup has arrived)."""
        self.check(self._lib.ckv_set_barrier_timeout_us(self.handle, int(us)))

    def policy(self) -> int:
        return int(self._lib.ckv_get_policy(self.handle))

    def set_kernel_timing(self, enable: bool):
        self.check(self._lib.ckv_set_kernel_timing(self.handle, int(bool(enable))))

    def set_kernel_timing_only(self, name: str | None):
        """Time only the kernel called ``name`` (None: every kernel)."""
        self.check(self._lib.ckv_set_kernel_timing_only(
            self.handle, None if name is None else name.encode()))

    def kernel_stats(self) -> dict:
        """{kernel name: (total ms, launches)} of the launches timed so far."""
        out, i = {}, 0
        name, ms, n = ctypes.c_char_p(), ctypes.c_double(), ctypes.c_int64()
        while self._lib.ckv_kernel_stats(self.handle, i, ctypes.byref(name), ctypes.byref(ms),
                                         ctypes.byref(n)) == 0:
            out[name.value.decode()] = (ms.value, n.value)
            i += 1
        return out

    def reset_kernel_stats(self):
        self.check(self._lib.ckv_reset_kernel_stats(self.handle))

    def last_error(self) -> str:
        return self._lib.ckv_last_error(self.handle).decode()

    def close(self):
        if getattr(self, "handle", None):
            self._lib.ckv_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- views

def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _check_bf16(t, name, ndim):
    if t.dtype != torch.bfloat16 or not t.is_cuda or t.dim() != ndim or t.stride(-1) != 1:
        raise ValueError(f"{name}: expected a cuda bfloat16 tensor of {ndim} dims with a contiguous last axis")


def kv_view(k, v, pos, n_tokens: int | None = None, slot=None) -> KVView:
    """k, v: [Hkv, S_cap, d] bf16 (same strides); pos: int32 [>= n_tokens].
    With ``slot`` (int32 [n_tokens], device), k and v are a paged pool of
    S_cap rows and token t lives in row slot[t]."""
    _check_bf16(k, "k", 3)
    _check_bf16(v, "v", 3)
    if k.shape != v.shape or k.stride() != v.stride():
        raise ValueError("k and v must have the same shape and strides")
    if pos.dtype != torch.int32 or not pos.is_cuda:
        raise ValueError("pos must be a cuda int32 tensor")
    if slot is not None:
        if slot.dtype != torch.int32 or not slot.is_cuda or not slot.is_contiguous():
            raise ValueError("slot must be a contiguous cuda int32 tensor")
        S = slot.numel() if n_tokens is None else int(n_tokens)
        if not 1 <= S <= slot.numel() or pos.numel() < S:
            raise ValueError("n_tokens out of range")
    else:
        S = k.shape[1] if n_tokens is None else int(n_tokens)
        if not 1 <= S <= k.shape[1] or pos.numel() < S:
            raise ValueError("n_tokens out of range")
    view = KVView(k.data_ptr(), v.data_ptr(), k.stride(0), k.stride(1), pos.data_ptr(), S,
                  k.shape[0], k.shape[2], slot.data_ptr() if slot is not None else None,
                  k.shape[1] if slot is not None else 0)
    view._keep = (k, v, pos, slot)   # the struct holds raw pointers: keep the tensors alive
    return view


def window_view(q, qpos, scale: float = 0.0) -> WindowView:
    """q: [Hq, W, d] bf16; qpos: int32 [W]."""
    _check_bf16(q, "q", 3)
    if qpos.dtype != torch.int32 or not qpos.is_cuda:
        raise ValueError("qpos must be a cuda int32 tensor")
    if qpos.numel() < q.shape[1]:
        raise ValueError("qpos shorter than the window")
    view = WindowView(q.data_ptr(), q.stride(0), q.stride(1), qpos.data_ptr(), q.shape[0],
                      q.shape[1], float(scale))
    view._keep = (q, qpos)
    return view


@dataclass
class Pages:
    """Host page list (kept alive alongside its ctypes view)."""
    start: np.ndarray
    len: np.ndarray

    def __post_init__(self):
        self.start = np.ascontiguousarray(self.start, dtype=np.int32)
        self.len = np.ascontiguousarray(self.len, dtype=np.int32)

    @property
    def n(self):
        return int(self.start.size)

    def view(self) -> PageList:
        return PageList(self.start.ctypes.data_as(_abi.c_i32p), self.len.ctypes.data_as(_abi.c_i32p),
                        self.n)


def cache_view(k, v, pos) -> CacheView:
    """k, v: [n_seq, n_layers, Hkv, capacity, d] bf16; pos: int32 [n_seq, >= capacity]."""
    _check_bf16(k, "k", 5)
    _check_bf16(v, "v", 5)
    if k.shape != v.shape or k.stride() != v.stride():
        raise ValueError("k and v must have the same shape and strides")
    if pos.dtype != torch.int32 or pos.dim() != 2 or pos.stride(1) != 1:
        raise ValueError("pos must be int32 [n_seq, capacity] with a contiguous last axis")
    s = k.stride()
    view = CacheView(k.data_ptr(), v.data_ptr(), s[0], s[1], s[2], s[3], pos.data_ptr(),
                     pos.stride(0), k.shape[0], k.shape[1], k.shape[2], k.shape[4], k.shape[3])
    view._keep = (k, v, pos)
    return view


def _f32(n, device, fill=None):
    t = torch.empty(n, dtype=torch.float32, device=device)
    if fill is not None:
        t.fill_(fill)
    return t


# ---------------------------------------------------------------- calls

def ckv_measure_page_effects(ctx: Context, kv: KVView, win: WindowView, pages: Pages, *,
                             R=None, R_head=None, o=None, lse=None, token_mass=None,
                             want=("R",), noalloc=False):
    """Window deletion effect of every page.  ``want`` names the optional
    outputs to allocate when not given: "R_head", "o", "lse", "token_mass".
    ``noalloc`` calls ckv_measure_page_effects_noalloc (the library allocates
    nothing; outputs are still allocated here unless given)."""
    dev = torch.device("cuda", ctx.device)
    Hq, W, d = win.n_q_heads, win.n_rows, kv.head_dim
    if R is None:
        R = _f32(max(pages.n, 1), dev)
    if R_head is None and "R_head" in want:
        R_head = _f32(max(pages.n * Hq, 1), dev)
    if o is None and "o" in want:
        o = _f32(Hq * W * d, dev)
    if lse is None and "lse" in want:
        lse = _f32(Hq * W, dev)
    if token_mass is None and "token_mass" in want:
        token_mass = _f32(kv.n_tokens, dev)
    pl = pages.view()
    fn = lib().ckv_measure_page_effects_noalloc if noalloc else lib().ckv_measure_page_effects
    ctx.check(fn(ctx.handle, ctypes.byref(kv), ctypes.byref(win), ctypes.byref(pl), _ptr(R),
                 _ptr(R_head), _ptr(o), _ptr(lse), _ptr(token_mass)))
    return dict(R=R[:pages.n], R_head=None if R_head is None else R_head[:pages.n * Hq].view(pages.n, Hq),
                o=None if o is None else o.view(Hq, W, d),
                lse=None if lse is None else lse.view(Hq, W), token_mass=token_mass)


def ckv_measure_page_effects_batch(ctx: Context, kvs, wins, pages, *, R=None, want=("R",)):
    """Problem i: kvs[i], wins[i], pages[i] (Pages).  Returns one dict per
    problem, as ckv_measure_page_effects does."""
    n = len(kvs)
    dev = torch.device("cuda", ctx.device)
    outs = []
    for i in range(n):
        Hq, W, d = wins[i].n_q_heads, wins[i].n_rows, kvs[i].head_dim
        np_ = pages[i].n
        outs.append(dict(
            R=R[i] if R is not None else _f32(max(np_, 1), dev),
            R_head=_f32(max(np_ * Hq, 1), dev) if "R_head" in want else None,
            o=_f32(Hq * W * d, dev) if "o" in want else None,
            lse=_f32(Hq * W, dev) if "lse" in want else None,
            token_mass=_f32(kvs[i].n_tokens, dev) if "token_mass" in want else None))
    kv_arr = (KVView * n)(*kvs)
    win_arr = (WindowView * n)(*wins)
    views = [p.view() for p in pages]
    pg_arr = (PageList * n)(*views)

    def ptrs(key):
        if all(o[key] is None for o in outs):
            return None
        return (ctypes.c_void_p * n)(*[(o[key].data_ptr() if o[key] is not None else 0) for o in outs])
    arrs = [ptrs(k) for k in ("R", "R_head", "o", "lse", "token_mass")]
    ctx.check(lib().ckv_measure_page_effects_batch(ctx.handle, n, kv_arr, win_arr, pg_arr, *arrs))
    res = []
    for i, o in enumerate(outs):
        np_, Hq, W, d = pages[i].n, wins[i].n_q_heads, wins[i].n_rows, kvs[i].head_dim
        res.append(dict(R=o["R"][:np_],
                        R_head=None if o["R_head"] is None else o["R_head"][:np_ * Hq].view(np_, Hq),
                        o=None if o["o"] is None else o["o"].view(Hq, W, d),
                        lse=None if o["lse"] is None else o["lse"].view(Hq, W),
                        token_mass=o["token_mass"]))
    return res


def ckv_measure_recorded(ctx: Context, kv: KVView, win: WindowView, pages: Pages, o, lse, *,
                         R=None, R_head=None, token_mass=None, want=("R",)):
    """Deletion effect of every page from recorded window outputs o [Hq, W, d]
    and log-sum-exp lse [Hq, W] (float32, device)."""
    dev = torch.device("cuda", ctx.device)
    Hq = win.n_q_heads
    if o.dtype != torch.float32 or lse.dtype != torch.float32 or not o.is_contiguous() or not lse.is_contiguous():
        raise ValueError("o and lse must be contiguous float32 tensors")
    if R is None:
        R = _f32(max(pages.n, 1), dev)
    if R_head is None and "R_head" in want:
        R_head = _f32(max(pages.n * Hq, 1), dev)
    if token_mass is None and "token_mass" in want:
        token_mass = _f32(kv.n_tokens, dev)
    pl = pages.view()
    ctx.check(lib().ckv_measure_recorded(ctx.handle, ctypes.byref(kv), ctypes.byref(win), ctypes.byref(pl),
                                         _ptr(o), _ptr(lse), _ptr(R), _ptr(R_head), _ptr(token_mass)))
    return dict(R=R[:pages.n], R_head=None if R_head is None else R_head[:pages.n * Hq].view(pages.n, Hq),
                token_mass=token_mass)


def ckv_pool_scores(ctx: Context, score, n_tokens, kernel: int = 7, mode: str = "max", out=None):
    """score: float32 [n_seq, stride] (device); n_tokens: ints per sequence."""
    if score.dtype != torch.float32 or score.dim() != 2 or score.stride(1) != 1:
        raise ValueError("score must be float32 [n_seq, stride] with a contiguous last axis")
    if out is None:
        out = torch.zeros_like(score)
    nt = np.ascontiguousarray(n_tokens, dtype=np.int32)
    ctx.check(lib().ckv_pool_scores(ctx.handle, _ptr(score), _ptr(out), score.shape[0], score.stride(0),
                                    nt.ctypes.data_as(_abi.c_i32p), int(kernel),
                                    {"max": _abi.POOL_MAX, "mean": _abi.POOL_MEAN}[mode]))
    return out


def ckv_classify_pages(ctx: Context, R_pre, R_post, thresholds: dict | None = None, *,
                       force=None, max_cand: int = 0):
    n = int(R_pre.numel())
    dev = R_pre.device
    th = dict(PAPER_THRESHOLDS)
    th.update(thresholds or {})
    t = Thresholds(th["tau_use"], th["tau_dead"], th["rho_use"], th["rho_dead"], th["tau_joint"])
    lam = torch.empty(max(n, 1), dtype=torch.uint8, device=dev)
    P_pre = _f32(max(n, 1), dev)
    P_post = _f32(max(n, 1), dev)
    cand = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
    n_cand = torch.empty(1, dtype=torch.int32, device=dev)     # written by the call
    ctx.check(lib().ckv_classify_pages(ctx.handle, n, _ptr(R_pre), _ptr(R_post), ctypes.byref(t),
                                       _ptr(force), int(max_cand), _ptr(lam), _ptr(P_pre),
                                       _ptr(P_post), _ptr(cand), _ptr(n_cand)))
    return dict(lam=lam[:n], P_pre=P_pre[:n], P_post=P_post[:n], cand=cand[:n], n_cand=n_cand)


def ckv_joint_test(ctx: Context, kv: KVView, win: WindowView, o, lse, pages: Pages, cand, n_cand,
                   max_cand: int, tau_joint: float = 0.01):
    dev = o.device
    accepted = torch.empty(max_cand, dtype=torch.uint8, device=dev)
    union_R = _f32(max_cand, dev)
    n_acc = torch.empty(1, dtype=torch.int32, device=dev)      # written by the call
    pl = pages.view()
    ctx.check(lib().ckv_joint_test(ctx.handle, ctypes.byref(kv), ctypes.byref(win), _ptr(o),
                                   _ptr(lse), ctypes.byref(pl), _ptr(cand), _ptr(n_cand),
                                   int(max_cand), float(tau_joint), _ptr(accepted), _ptr(union_R),
                                   _ptr(n_acc)))
    return dict(accepted=accepted, union_R=union_R, n_accepted=n_acc)


def ckv_select_and_compact(ctx: Context, k_in, v_in, pos_in, n_tokens, score, retired, pending,
                           pending_r_pre, *, budget: int, eta: float = 0.125,
                           max_pending_pages: int = 16, keep_recent: int = 0,
                           k_out=None, v_out=None, pos_out=None, token_state=None,
                           accepted=None, kept=None, n_kept=None, compact: bool = True):
    """k_in, v_in: [n_seq, n_layers, Hkv, capacity, d] bf16; pos_in: [n_seq, capacity] int32;
    n_tokens: host ints [n_seq]; score: [n_seq, stride] fp32; retired, pending: lists of
    Pages (one per sequence); pending_r_pre: list of fp32 device tensors (or None).
    accepted: optional list (one per sequence) of None or (Pages, cand, n_cand,
    accepted flags, max_cand) -- pages retired on the device by the joint test.
    compact=False runs the selection only (no output cache; k_in, v_in only
    give the shape)."""
    ns, L, H, cap, d = k_in.shape
    dev = k_in.device
    if not compact:
        k_out = v_out = pos_out = None
    elif k_out is None:
        k_out = torch.empty((ns, L, H, budget, d), dtype=torch.bfloat16, device=dev)
        v_out = torch.empty_like(k_out)
    if pos_out is None and compact:
        pos_out = torch.empty((ns, budget), dtype=torch.int32, device=dev)
    if kept is None:
        kept = torch.empty((ns, budget), dtype=torch.int32, device=dev)
    if n_kept is None:
        n_kept = torch.empty(ns, dtype=torch.int32, device=dev)   # written by the call
    cin = cache_view(k_in, v_in, pos_in)
    cout = cache_view(k_out, v_out, pos_out) if compact else None
    acc_arr, keep = None, []
    if accepted is not None:
        acc_arr = (AcceptedPages * ns)()
        for s_, e in enumerate(accepted):
            if e is None:
                continue
            pg, cand, ncand, flags, mc = e
            pl = pg.view()
            keep.append(pl)
            acc_arr[s_] = AcceptedPages(ctypes.cast(ctypes.pointer(pl), ctypes.c_void_p), _ptr(cand),
                                        _ptr(ncand), _ptr(flags), int(mc))
    nt = np.ascontiguousarray(n_tokens, dtype=np.int32)
    ret = (PageList * ns)(*[p.view() for p in retired])
    pen = (PageList * ns)(*[p.view() for p in pending])
    rptr = (ctypes.c_void_p * ns)(*[(r.data_ptr() if r is not None else 0) for r in pending_r_pre])
    b = Budget(int(budget), float(eta), int(max_pending_pages), int(keep_recent))
    ctx.check(lib().ckv_select_and_compact(
        ctx.handle, ctypes.byref(cin), nt.ctypes.data_as(_abi.c_i32p), _ptr(score),
        int(score.stride(0)), ret, pen, rptr, acc_arr, ctypes.byref(b),
        ctypes.byref(cout) if cout is not None else None, _ptr(kept),
        _ptr(n_kept), _ptr(token_state)))
    return dict(k=k_out, v=v_out, pos=pos_out, kept=kept, n_kept=n_kept)


# ---------------------------------------------------------------- lifecycle driver

def _np(ptr, n, dtype):
    if not ptr or n <= 0:
        return np.zeros(0, dtype)
    return np.ctypeslib.as_array(ptr, shape=(n,)).astype(dtype, copy=True)


class Agent:
    """The lifecycle driver of one agent episode (include/commitkv_agent.h,
    Algorithm 1).

    Contiguous (default): two cache buffers this object allocates,
    k, v [1, n_layers, Hkv, capacity, d] bf16 and pos [1, capacity] int32; a
    checkpoint compacts the cache into the other buffer.
    Paged (``paged=True``): one pool per layer, kp, vp [n_layers, Hkv,
    pool_rows, d] bf16 (``pool_rows`` defaults to the capacity), and a free
    list of rows standing in for a serving engine's block allocator; a
    checkpoint only re-indexes the agent's slot table and returns the rows of
    the dropped tokens to the free list.  ``row_seed`` shuffles the free list
    so that consecutive tokens land in scattered rows.

    ``append`` places the new tokens' keys, values and positions (a device
    copy) and reports them; ``commit``, ``post`` and ``checkpoint`` take the
    window's queries [Hq, W, d] (bf16, device) and positions (int32, device)
    and return the call's report as NumPy arrays."""

    def __init__(self, ctx: Context, n_layers: int, n_kv_heads: int, head_dim: int, capacity: int, *,
                 page_size: int, window: int, n_q_heads: int, budget: int, eta: float = 0.125,
                 max_pending_pages: int = 16, keep_recent: int = 0, max_scan_pages: int = 64,
                 checkpoint_every: int = 128, score_layer: int = 0, thresholds: dict | None = None,
                 report_detail: bool = False, pool_kernel: int = 0, pool_mode: str = "max",
                 paged: bool = False, pool_rows: int | None = None, row_seed: int | None = None):
        self.ctx = ctx
        self.paged = bool(paged)
        self.handle = None
        dev = torch.device("cuda", ctx.device)
        th = dict(PAPER_THRESHOLDS)
        th.update(thresholds or {})
        cfg = _abi.AgentConfig(page_size, window, n_q_heads, max_scan_pages, checkpoint_every,
                               score_layer, int(bool(report_detail)), Thresholds(**th),
                               Budget(budget, eta, max_pending_pages, keep_recent), int(pool_kernel),
                               {"max": _abi.POOL_MAX, "mean": _abi.POOL_MEAN}[pool_mode])
        h = ctypes.c_void_p()
        if self.paged:
            rows = capacity if pool_rows is None else int(pool_rows)
            shape = (n_layers, n_kv_heads, rows, head_dim)
            self.kp = torch.zeros(shape, dtype=torch.bfloat16, device=dev)
            self.vp = torch.zeros(shape, dtype=torch.bfloat16, device=dev)
            order = np.arange(rows)
            if row_seed is not None:
                order = np.random.default_rng(row_seed).permutation(rows)
            self.free = [int(r) for r in order[::-1]]      # pop() takes the next row
            kl, vl = self.kp[score_layer], self.vp[score_layer]
            self._pool = _abi.KVView(kl.data_ptr(), vl.data_ptr(), kl.stride(0), kl.stride(1), None, 0,
                                     n_kv_heads, head_dim, None, rows)
            ctx.check(lib().ckv_agent_create_paged(ctx.handle, ctypes.byref(self._pool), int(capacity),
                                                   ctypes.byref(cfg), ctypes.byref(h)))
        else:
            shape = (1, n_layers, n_kv_heads, capacity, head_dim)
            self.k = [torch.zeros(shape, dtype=torch.bfloat16, device=dev) for _ in range(2)]
            self.v = [torch.zeros(shape, dtype=torch.bfloat16, device=dev) for _ in range(2)]
            self.pos = [torch.zeros((1, capacity), dtype=torch.int32, device=dev) for _ in range(2)]
            self._views = [cache_view(self.k[i], self.v[i], self.pos[i]) for i in range(2)]
            ctx.check(lib().ckv_agent_create(ctx.handle, ctypes.byref(self._views[0]),
                                             ctypes.byref(self._views[1]), ctypes.byref(cfg), ctypes.byref(h)))
        self.handle = h

    def state(self):
        n, cur, dec = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64()
        self.ctx.check(lib().ckv_agent_state(self.handle, ctypes.byref(n), ctypes.byref(cur), ctypes.byref(dec)))
        return n.value, cur.value, dec.value

    def rows(self, which: str = "resident") -> np.ndarray:
        """"resident": pool rows of the resident tokens (paged); "freed": rows
        the last checkpoint released (paged); "pos": resident positions."""
        w = {"resident": 0, "freed": 1, "pos": 2}[which]
        n = ctypes.c_int32()
        self.ctx.check(lib().ckv_agent_rows(self.handle, w, None, 0, ctypes.byref(n)))
        out = np.zeros(max(n.value, 1), np.int32)
        self.ctx.check(lib().ckv_agent_rows(self.handle, w, out.ctypes.data_as(_abi.c_i32p), n.value,
                                            ctypes.byref(n)))
        return out[:n.value]

    def cache(self):
        """(k, v, pos, n_resident): k, v [n_layers, Hkv, >= n, d]; for a paged
        agent a gathered copy of the resident rows."""
        n, cur, _ = self.state()
        if self.paged:
            idx = torch.from_numpy(self.rows("resident").astype(np.int64)).to(self.kp.device)
            pos = torch.from_numpy(self.rows("pos")).to(self.kp.device)
            return self.kp[:, :, idx], self.vp[:, :, idx], pos, n
        return self.k[cur][0], self.v[cur][0], self.pos[cur][0], n

    def append(self, kind: int, k, v, pos, decoded: bool, begins_event: bool = True) -> int:
        """k, v: [n_layers, Hkv, n, d] bf16 (device); pos: host int array [n].
        Returns the CKV_DUE_* flags."""
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        n_tok = int(pos.size)
        n, cur, _ = self.state()
        due = ctypes.c_int32()
        if self.paged:
            if n_tok > len(self.free):
                raise CKVError(_abi.CKV_ERR_SHAPE, "pool has no free rows left")
            rows = np.array([self.free.pop() for _ in range(n_tok)], np.int32)
            if n_tok:
                idx = torch.from_numpy(rows.astype(np.int64)).to(self.kp.device)
                self.kp.index_copy_(2, idx, k)
                self.vp.index_copy_(2, idx, v)
            try:
                self.ctx.check(lib().ckv_agent_append_rows(
                    self.handle, int(kind), pos.ctypes.data_as(_abi.c_i32p), rows.ctypes.data_as(_abi.c_i32p),
                    n_tok, int(bool(decoded)), int(bool(begins_event)), ctypes.byref(due)))
            except CKVError:
                self.free.extend(rows[::-1].tolist())
                raise
            return due.value
        if n + n_tok > self.k[cur].shape[3]:
            raise CKVError(_abi.CKV_ERR_SHAPE, "cache buffer capacity exceeded")
        if n_tok:
            self.k[cur][0, :, :, n:n + n_tok].copy_(k)
            self.v[cur][0, :, :, n:n + n_tok].copy_(v)
            self.pos[cur][0, n:n + n_tok].copy_(torch.from_numpy(pos))
        self.ctx.check(lib().ckv_agent_append(self.handle, int(kind), pos.ctypes.data_as(_abi.c_i32p), n_tok,
                                              int(bool(decoded)), int(bool(begins_event)), ctypes.byref(due)))
        return due.value

    def commit(self, q, qpos):
        w = window_view(q, qpos)
        self.ctx.check(lib().ckv_agent_commit(self.handle, ctypes.byref(w)))
        return self.report()

    def post(self, q, qpos):
        w = window_view(q, qpos)
        self.ctx.check(lib().ckv_agent_post(self.handle, ctypes.byref(w)))
        return self.report()

    def checkpoint(self, q, qpos):
        w = window_view(q, qpos)
        c = ctypes.c_int32()
        self.ctx.check(lib().ckv_agent_checkpoint(self.handle, ctypes.byref(w), ctypes.byref(c)))
        if self.paged and c.value:
            self.free.extend(self.rows("freed").tolist())
        return self.report()

    def report(self) -> dict:
        r = _abi.AgentReport()
        self.ctx.check(lib().ckv_agent_last_report(self.handle, ctypes.byref(r)))
        n, nc = r.n_pages, r.n_cand
        return dict(op=r.op, pages=list(zip(_np(r.page_start, n, np.int64).tolist(),
                                            _np(r.page_len, n, np.int64).tolist())),
                    R_pre=_np(r.r_pre, n, np.float32), R_post=_np(r.r_post, n, np.float32),
                    lam=_np(r.lambda_, n, np.uint8), cand=_np(r.cand, nc, np.int64),
                    accepted=_np(r.accepted, nc, np.uint8), union_R=_np(r.union_r, nc, np.float32),
                    n_accepted=r.n_accepted, compacted=bool(r.compacted), n_before=r.n_before,
                    kept=_np(r.kept, r.n_kept, np.int64), score=_np(r.score, r.n_before, np.float32))

    def pages(self, which: str):
        """"pending" -> [(start, len, R-)], "retired" -> [(start, len)] (absolute positions)."""
        w = {"pending": 0, "retired": 1}[which]
        n = ctypes.c_int32()
        self.ctx.check(lib().ckv_agent_pages(self.handle, w, None, None, None, 0, ctypes.byref(n)))
        m = n.value
        st = np.zeros(max(m, 1), np.int32)
        ln = np.zeros(max(m, 1), np.int32)
        val = np.zeros(max(m, 1), np.float32)
        self.ctx.check(lib().ckv_agent_pages(self.handle, w, st.ctypes.data_as(_abi.c_i32p),
                                             ln.ctypes.data_as(_abi.c_i32p), val.ctypes.data_as(_abi.c_f32p),
                                             m, ctypes.byref(n)))
        if w == 0:
            return [(int(a), int(b), float(c)) for a, b, c in zip(st[:m], ln[:m], val[:m])]
        return [(int(a), int(b)) for a, b in zip(st[:m], ln[:m])]

    def close(self):
        if getattr(self, "handle", None):
            lib().ckv_agent_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
