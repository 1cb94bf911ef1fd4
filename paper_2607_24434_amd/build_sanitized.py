"""Builds the expert cache's host code with AddressSanitizer and UBSan, CPU only.

The expert cache (``csrc/cache.cpp``) is plain host bookkeeping around HIP
copies.  With fake copies (``de_cache_cfg.fake_copies = 1``) it makes no HIP
call at all and moves slot contents with ``memcpy``, so its whole state
machine can run on a machine without a GPU.  This script compiles that file
and the return-code strings with the host compiler under
``-fsanitize=address,undefined`` into a library that exports only the cache's
entry points.  ``paper_2607_24434_amd._lib`` loads it in place of the full
library when ``DE_LIBRARY`` names it; the cache tests then run under the
sanitizers (see ``tests/test_cache_sanitized.py``).

Usage: python paper_2607_24434_amd/build_sanitized.py   (prints the library path)
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(ROOT, "_build", "host_sanitized")
LIB = os.path.join(OUT_DIR, "libdraftexpert_cache_sanitized.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CXX = os.environ.get("HOST_CXX", "g++")
SOURCES = ["cache.cpp", "errors.cpp"]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def runtime_preload() -> str:
    """Path of the compiler's ASan runtime, which must be the first library
    loaded into a process (Python itself is not built with it)."""
    r = subprocess.run([CXX, "-print-file-name=libasan.so"], capture_output=True, text=True, check=True)
    path = r.stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError(f"{CXX} has no AddressSanitizer runtime")
    return path


def build() -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    cmd = [CXX, "-std=c++17", "-O1", "-g", "-fPIC", "-shared", *SAN, "-Wall",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I",
           os.path.join(ROCM, "include"), *[os.path.join(CSRC, s) for s in SOURCES],
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-o", LIB + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("command failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build())
    sys.exit(0)
