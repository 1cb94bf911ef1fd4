"""Builds the fills of the synthetic streams: libdesynth.so (gfx950) and libdesynth_cpu.so (gcc)."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libdesynth.so")
CPU_LIB = os.path.join(HERE, "libdesynth_cpu.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           os.path.join(HERE, "csrc", "synth_fill.hip"), "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(" ".join(cmd) + "\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    tmp = CPU_LIB + ".tmp"
    cmd = ["gcc", "-O3", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off",
           os.path.join(HERE, "csrc", "synth_cpu.c"), "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(" ".join(cmd) + "\n" + r.stdout + r.stderr)
    os.replace(tmp, CPU_LIB)
    if verbose:
        print("built", LIB, CPU_LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
