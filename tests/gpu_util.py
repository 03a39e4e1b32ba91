"""Helpers shared by the GPU parity tests (inputs to device, parity checks)."""
import numpy as np
import torch

import oracle as O

REL_TOL = 2e-3      # score tolerance for bf16 inputs with fp32 accumulation
ABS_FLOOR = 1e-6


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def dev_i32(x) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


class LayerOnDevice:
    def __init__(self, L):
        self.L = L
        self.k = dev_bf16(L.k)
        self.v = dev_bf16(L.v)
        self.pos = dev_i32(L.pos)
        self.q_pre = dev_bf16(L.q_pre)
        self.q_post = dev_bf16(L.q_post)
        self.qpos_pre = dev_i32(L.qpos_pre)
        self.qpos_post = dev_i32(L.qpos_post)


def assert_scores_close(got, want, what="R", rel=REL_TOL, floor=ABS_FLOOR):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    inf_g, inf_w = np.isinf(got), np.isinf(want)
    bad_inf = np.flatnonzero(inf_g != inf_w)
    assert bad_inf.size == 0, f"{what}: inf mismatch at {bad_inf[:10]} got {got.flat[bad_inf[:5]]} want {want.flat[bad_inf[:5]]}"
    fin = ~inf_w
    err = np.abs(got[fin] - want[fin])
    lim = rel * np.maximum(want[fin], floor)
    bad = np.flatnonzero(err > lim)
    rel_err = err / np.maximum(want[fin], floor)
    if rel_err.size:
        print(f"[parity] {what}: worst relative error {rel_err.max():.3g} over {rel_err.size} values", flush=True)
    if bad.size:
        i = int(np.argmax(rel_err))
        raise AssertionError(f"{what}: {bad.size}/{fin.sum()} outside {rel} relative; worst got "
                             f"{got[fin][i]!r} want {want[fin][i]!r} (rel {rel_err[i]:.3g})")


def oracle_pass(L, which, method="closed"):
    """Oracle R, R_h for the pre (prefix cache) or post (full cache) window."""
    if which == "pre":
        S = L.layout.s_pre
        return O.page_effects(L.k[:, :S], L.v[:, :S], L.pos[:S], L.q_pre, L.qpos_pre, L.pages,
                              method=method)
    return O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, method=method)
