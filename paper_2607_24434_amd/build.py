"""Builds libdraftexpert.so in-tree with hipcc for gfx950.

Usage: python paper_2607_24434_amd/build.py   (runs without importing the package,
whose import loads the library this script produces).
Every source compiles to its own object under _build/ in parallel, then one
shared library is linked next to this file.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libdraftexpert.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["api.cpp", "errors.cpp", "model.cpp", "cache.cpp", "router_topk.hip", "grouped_swiglu.hip", "glue.hip",
           "truncation.hip", "distill.hip", "noalloc.hip", "draft_persistent.hip", "rowdot_mfma.hip",
           "verify_fused.hip"]

# Packed fp32 instructions are disabled for every device compile; the host
# pass warns that it does not know the feature, which is harmless.
HIP_FLAGS = [
    "-x", "hip", f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
    "-I", os.path.join(ROOT, "include"),
]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("command failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r


def build(verbose: bool = False, extra_flags=None) -> str:
    bdir = os.path.join(ROOT, "_build", "draftexpert")
    os.makedirs(bdir, exist_ok=True)
    flags = HIP_FLAGS + list(extra_flags or [])

    def compile_one(src):
        obj = os.path.join(bdir, os.path.splitext(src)[0] + ".o")
        _run([HIPCC, *flags, "-c", os.path.join(CSRC, src), "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True, extra_flags=sys.argv[1:])
