"""The tooling builds on the GPU: the device-check library (CKV_DEBUG)
computes what the release library computes and none of its bounds checks
fires on the hot path, and the host-sanitizer build runs every C ABI entry
point clean under AddressSanitizer and UndefinedBehaviorSanitizer."""
import os
import subprocess

import numpy as np
import pytest
import torch

import paper_2608_07855_amd as P
from paper_2608_07855_amd import _abi, build
from synth import WORKLOADS, make_layer

from .gpu_util import dev_bf16, dev_i32

pytestmark = pytest.mark.gpu


def _hot_path(L, w):
    """Pre and post measurement, classification, joint test, selection and
    compaction on one layer; every output as numpy."""
    ctx = P.Context(0)
    try:
        k, v, pos = dev_bf16(L.k), dev_bf16(L.v), dev_i32(L.pos)
        pages = P.Pages(L.layout.page_start, L.layout.page_len)
        kv_pre = P.kv_view(k, v, pos, L.layout.s_pre)
        kv_post = P.kv_view(k, v, pos)
        win_pre = P.window_view(dev_bf16(L.q_pre), dev_i32(L.qpos_pre))
        win_post = P.window_view(dev_bf16(L.q_post), dev_i32(L.qpos_post))
        pre = P.ckv_measure_page_effects(ctx, kv_pre, win_pre, pages, want=("R", "R_head"))
        post = P.ckv_measure_page_effects(ctx, kv_post, win_post, pages,
                                          want=("R", "R_head", "o", "lse", "token_mass"))
        force = torch.zeros(len(L.layout.page_start), dtype=torch.uint8, device="cuda")
        force[::5] = 1
        cl = P.ckv_classify_pages(ctx, pre["R"], post["R"], force=force)
        jt = P.ckv_joint_test(ctx, kv_post, win_post, post["o"], post["lse"], pages, cl["cand"], cl["n_cand"],
                              len(L.layout.page_start))
        pend = L.layout.pending_idx
        sel = P.ckv_select_and_compact(
            ctx, k[None, None], v[None, None], pos[None], [w.n_tokens], post["token_mass"][None],
            [P.Pages([], [])], [P.Pages(L.layout.page_start[pend], L.layout.page_len[pend])],
            [pre["R"][torch.from_numpy(pend).cuda()].contiguous()],
            budget=w.budget, eta=w.eta, max_pending_pages=w.max_pending_pages, keep_recent=w.window)
        ctx.sync()
        out = {f"pre_{n}": pre[n] for n in ("R", "R_head")}
        out.update({f"post_{n}": post[n] for n in ("R", "R_head", "o", "lse", "token_mass")})
        out.update(lam=cl["lam"], cand=cl["cand"], n_cand=cl["n_cand"], acc=jt["accepted"],
                   union=jt["union_R"], n_acc=jt["n_accepted"])
        out.update({f"sel_{n}": sel[n] for n in sel if torch.is_tensor(sel[n])})
        # bf16 tensors (compacted keys and values) compared by their bits
        return {n: (t.view(torch.int16) if t.dtype == torch.bfloat16 else t).detach().cpu().numpy()
                for n, t in out.items()}
    finally:
        ctx.close()


@pytest.mark.parametrize("seed", [0, 1])
def test_device_check_build_matches_release(seed):
    if not os.path.exists(_abi.DEBUG_LIB_PATH):
        pytest.fail("libcommitkv_debug.so is not built (python -m paper_2608_07855_amd.build all)")
    name = "tiny"
    w = WORKLOADS[name]
    L = make_layer(w, seed=seed)
    print(f"[tools] release path on {name}", flush=True)
    rel = _hot_path(L, w)
    saved = _abi._lib
    try:
        _abi._lib = _abi.load(_abi.DEBUG_LIB_PATH)
        assert P.lib().ckv_build_flags() == _abi.BUILD_DEVICE_CHECKS
        print(f"[tools] device-check path on {name}", flush=True)
        dbg = _hot_path(L, w)   # a fired check raises CKVError (CKV_ERR_DEVICE_CHECK) here
    finally:
        _abi._lib = saved
    assert rel.keys() == dbg.keys()
    for n in rel:
        a, b = rel[n], dbg[n]
        assert a.shape == b.shape, n
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8)) or np.allclose(a, b, rtol=1e-6, atol=0,
                                                                                 equal_nan=True), n


def test_host_sanitizer_driver():
    if not os.path.exists(build.DRIVER):
        pytest.fail("the sanitizer driver is not built (python -m paper_2608_07855_amd.build asan)")
    env = dict(os.environ)
    # the GPU runtime maps memory where AddressSanitizer would otherwise
    # protect its shadow gap; the runtime's own allocations are not leaks
    env["ASAN_OPTIONS"] = "protect_shadow_gap=0:detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    print("[tools] sanitizer driver", flush=True)
    r = subprocess.run([build.DRIVER], env=env, capture_output=True, text=True, timeout=300)
    text = r.stdout + r.stderr
    print(text[-3000:], flush=True)
    assert "AddressSanitizer" not in text and "runtime error" not in text
    assert r.returncode == 0, text[-2000:]
    assert "[driver] ok" in r.stdout
