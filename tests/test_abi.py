"""The C-ABI library builds, loads and exports every entry point of include/*.h
(CPU only: nothing here launches GPU work)."""
import ctypes
import glob
import os
import re

import pytest

from paper_2608_07855_amd import _abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[\w\s\*]+?\b(ckv_\w+)\s*\(", text, flags=re.M):
            names.add(m.group(1))
    return names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_abi.LIB_PATH):
        from paper_2608_07855_amd import build
        build.build()
    return ctypes.CDLL(_abi.LIB_PATH)


def test_header_declares_the_four_calls():
    d = _declared()
    for name in ("ckv_measure_page_effects", "ckv_classify_pages", "ckv_joint_test",
                 "ckv_select_and_compact"):
        assert name in d


def test_every_declared_symbol_is_exported(lib):
    missing = [n for n in sorted(_declared()) if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_symbol():
    assert set(_abi.SIGNATURES) == _declared()


def test_version_and_null_handling(lib):
    L = _abi.load()
    v = L.ckv_version()
    assert v == (0 << 16) | (1 << 8) | 0
    # NULL context / arguments are rejected on the host without touching a device
    assert L.ckv_sync(None) == _abi.CKV_ERR_ARG
    assert L.ckv_destroy(None) == _abi.CKV_ERR_ARG
    assert L.ckv_create(None, 0, None) == _abi.CKV_ERR_ARG
    assert L.ckv_last_error(None) == b"NULL context"
    assert L.ckv_workspace_bytes(None) == 0


def test_struct_layouts_match_header():
    # field order and sizes of the views as the header declares them
    assert ctypes.sizeof(_abi.KVView) == 8 + 8 + 8 + 8 + 8 + 4 * 3 + 4
    assert ctypes.sizeof(_abi.WindowView) == 8 + 8 + 8 + 8 + 4 * 3 + 4
    assert ctypes.sizeof(_abi.PageList) == 8 + 8 + 4 + 4
    assert ctypes.sizeof(_abi.Thresholds) == 20
    assert ctypes.sizeof(_abi.Budget) == 16
    assert ctypes.sizeof(_abi.CacheView) == 8 * 2 + 8 * 4 + 8 + 8 + 4 * 5 + 4


def test_policy_bits_match_header(lib):
    text = open(os.path.join(ROOT, "include", "commitkv.h")).read()
    hdr = {m.group(1).lower(): int(m.group(2))
           for m in re.finditer(r"CKV_POLICY_(NO_\w+)\s*=\s*(\d+)", text)}
    assert hdr == _abi.POLICY_BITS
    L = _abi.load()
    assert L.ckv_set_policy(None, 1) == _abi.CKV_ERR_ARG
    assert L.ckv_get_policy(None) == 0
