"""ctypes declarations of include/commitkv.h, include/commitkv_agent.h and the
library loader.

The library is the in-tree ``libcommitkv.so`` built by
``python -m paper_2608_07855_amd.build``.  There is no fallback: if the
library is missing, loading raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcommitkv.so")
# the same library built with device bounds checks (CKV_DEBUG)
DEBUG_LIB_PATH = os.path.join(_HERE, "libcommitkv_debug.so")
BUILD_DEVICE_CHECKS = 1

CKV_OK = 0
CKV_ERR_ARG = -1
CKV_ERR_SHAPE = -2
CKV_ERR_BUDGET = -3
CKV_ERR_UNSUPPORTED = -4
CKV_ERR_NOMEM = -5
CKV_ERR_HIP = -6
CKV_ERR_NONFINITE = -7
CKV_ERR_DEVICE_CHECK = -8
STATUS_NAMES = {0: "CKV_OK", -1: "CKV_ERR_ARG", -2: "CKV_ERR_SHAPE", -3: "CKV_ERR_BUDGET",
                -4: "CKV_ERR_UNSUPPORTED", -5: "CKV_ERR_NOMEM", -6: "CKV_ERR_HIP",
                -7: "CKV_ERR_NONFINITE", -8: "CKV_ERR_DEVICE_CHECK"}
MAX_PAGE_LEN = 64
# ckv_policy_flag: component switches of the Sec. 4.4 ablation variants
POLICY_NO_PRECOMMIT = 1
POLICY_NO_PERCENTILE = 2
POLICY_NO_JOINT = 4
POLICY_NO_PROTECTION = 8
POLICY_NO_LIFECYCLE = 16
POLICY_BITS = {"no_precommit": POLICY_NO_PRECOMMIT, "no_percentile": POLICY_NO_PERCENTILE,
               "no_joint": POLICY_NO_JOINT, "no_protection": POLICY_NO_PROTECTION,
               "no_lifecycle": POLICY_NO_LIFECYCLE}

c_i32p = ctypes.POINTER(ctypes.c_int32)
c_f32p = ctypes.POINTER(ctypes.c_float)
c_u8p = ctypes.POINTER(ctypes.c_uint8)
c_u16p = ctypes.POINTER(ctypes.c_uint16)


class KVView(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("head_stride", ctypes.c_int64), ("tok_stride", ctypes.c_int64),
                ("pos", ctypes.c_void_p), ("n_tokens", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("slot", ctypes.c_void_p), ("pool_rows", ctypes.c_int32)]


class WindowView(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("head_stride", ctypes.c_int64),
                ("row_stride", ctypes.c_int64), ("qpos", ctypes.c_void_p),
                ("n_q_heads", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("scale", ctypes.c_float)]


class PageList(ctypes.Structure):
    _fields_ = [("start", c_i32p), ("len", c_i32p), ("n_pages", ctypes.c_int32)]


class Thresholds(ctypes.Structure):
    _fields_ = [("tau_use", ctypes.c_float), ("tau_dead", ctypes.c_float),
                ("rho_use", ctypes.c_float), ("rho_dead", ctypes.c_float),
                ("tau_joint", ctypes.c_float)]


class Budget(ctypes.Structure):
    _fields_ = [("budget", ctypes.c_int32), ("eta", ctypes.c_float),
                ("max_pending_pages", ctypes.c_int32), ("keep_recent", ctypes.c_int32)]


class CacheView(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("seq_stride", ctypes.c_int64), ("layer_stride", ctypes.c_int64),
                ("head_stride", ctypes.c_int64), ("tok_stride", ctypes.c_int64),
                ("pos", ctypes.c_void_p), ("pos_seq_stride", ctypes.c_int64),
                ("n_seq", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("capacity", ctypes.c_int32)]


class AcceptedPages(ctypes.Structure):
    _fields_ = [("pages", ctypes.c_void_p), ("cand", ctypes.c_void_p), ("n_cand", ctypes.c_void_p),
                ("accepted", ctypes.c_void_p), ("max_cand", ctypes.c_int32)]


POOL_MAX, POOL_MEAN = 0, 1

# ckv_event_kind and the due flags of include/commitkv_agent.h
EVENT_REASONING, EVENT_TOOL_CALL, EVENT_OBSERVATION, EVENT_PROMPT, EVENT_ANSWER = range(5)
DUE_POST = 1
DUE_CHECKPOINT = 2


class AgentConfig(ctypes.Structure):
    _fields_ = [("page_size", ctypes.c_int32), ("window", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("max_scan_pages", ctypes.c_int32),
                ("checkpoint_every", ctypes.c_int32), ("score_layer", ctypes.c_int32),
                ("report_detail", ctypes.c_int32), ("thresholds", Thresholds),
                ("budget", Budget), ("pool_kernel", ctypes.c_int32), ("pool_mode", ctypes.c_int32)]


class AgentReport(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("n_pages", ctypes.c_int32),
                ("page_start", c_i32p), ("page_len", c_i32p), ("r_pre", c_f32p),
                ("r_post", c_f32p), ("lambda_", c_u8p), ("n_cand", ctypes.c_int32),
                ("cand", c_i32p), ("accepted", c_u8p), ("union_r", c_f32p),
                ("n_accepted", ctypes.c_int32), ("compacted", ctypes.c_int32),
                ("n_before", ctypes.c_int32), ("n_kept", ctypes.c_int32),
                ("kept", c_i32p), ("score", c_f32p)]


# name -> (restype, argtypes): every entry point of include/*.h
SIGNATURES = {
    "ckv_create": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int, ctypes.c_void_p]),
    "ckv_destroy": (ctypes.c_int, [ctypes.c_void_p]),
    "ckv_set_stream": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p]),
    "ckv_sync": (ctypes.c_int, [ctypes.c_void_p]),
    "ckv_last_error": (ctypes.c_char_p, [ctypes.c_void_p]),
    "ckv_version": (ctypes.c_uint32, []),
    "ckv_build_flags": (ctypes.c_uint32, []),
    "ckv_set_workspace_limit": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t]),
    "ckv_workspace_bytes": (ctypes.c_size_t, [ctypes.c_void_p]),
    "ckv_set_policy": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_uint32]),
    "ckv_get_policy": (ctypes.c_uint32, [ctypes.c_void_p]),
    "ckv_set_barrier_timeout_us": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64]),
    "ckv_set_kernel_timing": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int]),
    "ckv_set_kernel_timing_only": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_char_p]),
    "ckv_kernel_stats": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32,
                                        ctypes.POINTER(ctypes.c_char_p),
                                        ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int64)]),
    "ckv_reset_kernel_stats": (ctypes.c_int, [ctypes.c_void_p]),
    "ckv_measure_page_effects": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.POINTER(KVView), ctypes.POINTER(WindowView),
        ctypes.POINTER(PageList), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p]),
    "ckv_measure_page_effects_noalloc": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.POINTER(KVView), ctypes.POINTER(WindowView),
        ctypes.POINTER(PageList), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p]),
    "ckv_measure_page_effects_batch": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(KVView), ctypes.POINTER(WindowView),
        ctypes.POINTER(PageList), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p]),
    "ckv_measure_recorded": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.POINTER(KVView), ctypes.POINTER(WindowView),
        ctypes.POINTER(PageList), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p]),
    "ckv_classify_pages": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.POINTER(Thresholds), ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "ckv_joint_test": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.POINTER(KVView), ctypes.POINTER(WindowView),
        ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(PageList), ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p]),
    "ckv_pool_scores": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                       ctypes.c_int64, c_i32p, ctypes.c_int32, ctypes.c_int32]),
    "ckv_select_and_compact": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.POINTER(CacheView), c_i32p, ctypes.c_void_p,
        ctypes.c_int64, ctypes.POINTER(PageList), ctypes.POINTER(PageList),
        ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(AcceptedPages), ctypes.POINTER(Budget),
        ctypes.POINTER(CacheView), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "ckv_agent_create": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(CacheView),
                                        ctypes.POINTER(CacheView), ctypes.POINTER(AgentConfig),
                                        ctypes.POINTER(ctypes.c_void_p)]),
    "ckv_agent_destroy": (ctypes.c_int, [ctypes.c_void_p]),
    "ckv_agent_append": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, c_i32p, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_int32, c_i32p]),
    "ckv_agent_commit": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(WindowView)]),
    "ckv_agent_post": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(WindowView)]),
    "ckv_agent_checkpoint": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(WindowView), c_i32p]),
    "ckv_agent_state": (ctypes.c_int, [ctypes.c_void_p, c_i32p, c_i32p,
                                       ctypes.POINTER(ctypes.c_int64)]),
    "ckv_agent_last_report": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(AgentReport)]),
    "ckv_agent_pages": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, c_i32p, c_i32p, c_f32p,
                                       ctypes.c_int32, c_i32p]),
    "ckv_agent_create_paged": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(KVView), ctypes.c_int32,
                                              ctypes.POINTER(AgentConfig), ctypes.POINTER(ctypes.c_void_p)]),
    "ckv_agent_append_rows": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, c_i32p, c_i32p, ctypes.c_int32,
                                             ctypes.c_int32, ctypes.c_int32, c_i32p]),
    "ckv_agent_rows": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, c_i32p, ctypes.c_int32, c_i32p]),
}

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libcommitkv.so and declare its entry points (raises if absent)."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise OSError(f"{path} not found: build it with `python -m paper_2608_07855_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path == LIB_PATH:
        _lib = lib
    return lib
