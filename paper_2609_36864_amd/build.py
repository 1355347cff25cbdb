"""Build libhdl.so (all HIP kernels + the C ABI) for gfx950 with hipcc.

Usage: python -m paper_2609_36864_amd.build   (or build_library() from Python).
The library is written next to this file so it travels with the source tree.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
LIB_PATH = os.path.join(PKG_DIR, "libhdl.so")
CEILING_PATH = os.path.join(PKG_DIR, "mfma_ceiling")
ARCH = "gfx950"

HIP_FLAGS = [
    "-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function", "-Werror=uninitialized",
    # keep packed-fp32 VALU instructions out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def sources():
    return sorted(glob.glob(os.path.join(PKG_DIR, "csrc", "*.hip")))


def _hipcc(args, verbose):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    cmd = [hipcc, *args]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature and says so; drop
    # that one harmless line from what we show
    noise = "'-packed-fp32-ops' is not a recognized feature"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def build_ceiling_tool(verbose: bool = False) -> str:
    """The MFMA ceiling microbenchmark used by bench.py --mfma-ceiling."""
    tmp = CEILING_PATH + ".tmp"
    flags = [f for f in HIP_FLAGS if f not in ("-fPIC", "-shared")]
    _hipcc([*flags, os.path.join(PKG_DIR, "csrc", "tools", "mfma_ceiling.hip"), "-o", tmp], verbose)
    os.replace(tmp, CEILING_PATH)
    return CEILING_PATH


ABI_CHECK_PATH = os.path.join(PKG_DIR, "abi_check")


def build_abi_check(verbose: bool = False) -> str:
    """A native C++ consumer of the C ABI (no Python): links libhdl.so,
    which must be built first; finds it next to itself at run time."""
    tmp = ABI_CHECK_PATH + ".tmp"
    _hipcc(["-O2", "-std=c++17", "-Wall", "-I", os.path.join(ROOT, "include"),
            os.path.join(PKG_DIR, "csrc", "tools", "abi_check.cpp"),
            "-L", PKG_DIR, "-lhdl", "-Wl,-rpath,$ORIGIN", "-o", tmp], verbose)
    os.replace(tmp, ABI_CHECK_PATH)
    return ABI_CHECK_PATH


def build_library(verbose: bool = False) -> str:
    tmp = LIB_PATH + ".tmp"
    _hipcc([*HIP_FLAGS, "-I", os.path.join(ROOT, "include"), *sources(), "-o", tmp], verbose)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build_library(verbose=True))
    print(build_ceiling_tool(verbose=True))
    print(build_abi_check(verbose=True))
