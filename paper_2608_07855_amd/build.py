"""Build the library (gfx950 only) with hipcc, in-tree.

    python -m paper_2608_07855_amd.build [-v] [release|debug|asan|all]

release  paper_2608_07855_amd/libcommitkv.so, the product.
debug    paper_2608_07855_amd/libcommitkv_debug.so: the same sources with
         -DCKV_DEBUG, i.e. device bounds checks (see ckv_build_flags in
         include/commitkv.h).
asan     paper_2608_07855_amd/libcommitkv_asan.so: host code built with
         AddressSanitizer and UndefinedBehaviorSanitizer (device code as in
         release), and _build/asan/abi_driver, a program that runs every C
         ABI entry point (tests/native/abi_driver.cpp) against it.

Objects go to ``paper_2608_07855_amd/_build/<variant>``.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["api.cpp", "agent.cpp", "measure.hip", "recorded.hip", "classify.hip", "joint.hip", "select.hip"]

COMMON = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-result",
    # packed fp32 instructions stay off on this target
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]
# sanitizers on the host side only (device code is never built with them)
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]
VARIANTS = {
    "release": ("libcommitkv.so", []),
    "debug": ("libcommitkv_debug.so", ["-DCKV_DEBUG"]),
    "asan": ("libcommitkv_asan.so", HOST_SANITIZE),
}
LIB = os.path.join(PKG, VARIANTS["release"][0])
DRIVER = os.path.join(BUILD_DIR, "asan", "abi_driver")
# roctx ranges (rocprofiler-sdk's roctx library, part of every ROCm 7 install)
LINK_LIBS = ["-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"]


def _run(cmd, verbose, what):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(line for line in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"{what} failed:\n{msgs}")
    if verbose and msgs.strip():
        print(msgs, flush=True)


def _compile(src: str, out_dir: str, flags, verbose: bool) -> str:
    obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
    _run([HIPCC, "-x", "hip", *COMMON, *flags, "-c", os.path.join(CSRC, src), "-o", obj], verbose,
         f"hipcc on {src}")
    return obj


def build(verbose: bool = False, variant: str = "release") -> str:
    """Compile and link one variant; returns the library's path."""
    name, flags = VARIANTS[variant]
    out_dir = os.path.join(BUILD_DIR, variant)
    os.makedirs(out_dir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(lambda s: _compile(s, out_dir, flags, verbose), SOURCES))
    lib = os.path.join(PKG, name)
    tmp = lib + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs, *LINK_LIBS], verbose,
         f"link of {name}")
    os.replace(tmp, lib)
    if variant == "asan":
        # the driver carries the sanitizer runtimes; it finds the library
        # two directories up from itself
        _run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-std=c++17", "-Wall",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *HOST_SANITIZE,
              "-I", INCLUDE, os.path.join(ROOT, "tests", "native", "abi_driver.cpp"), "-o", DRIVER,
              "-L", PKG, "-lcommitkv_asan", "-Wl,-rpath,$ORIGIN/../..", *LINK_LIBS], verbose,
             "abi_driver build")
    return lib


def build_all(verbose: bool = False) -> list:
    return [build(verbose, v) for v in VARIANTS]


if __name__ == "__main__":
    args = [a for a in sys.argv[1:] if a != "-v"]
    which = args[0] if args else "release"
    verbose = "-v" in sys.argv[1:]
    if which == "all":
        print("\n".join(build_all(verbose)))
    else:
        print(build(verbose, which))
