"""The expert cache's host code under AddressSanitizer and UBSan, on the CPU.

``paper_2607_24434_amd/build_sanitized.py`` compiles ``csrc/cache.cpp`` with
the host compiler and ``-fsanitize=address,undefined`` into a library that
exports only the cache's entry points.  ``tests/test_cache.py`` then runs in a
child process against that library (``DE_LIBRARY``), with the ASan runtime
preloaded, over fake copies: every bookkeeping case, the comparison with the
simulation on random request sequences and the argument errors.  Any
out-of-bounds access, use after free or undefined behaviour in the cache's
host code ends the child with the sanitizer's report and fails this test.
The child runs without output capture, so that a sanitizer report, written
to the file descriptor as the process dies, reaches this test's output.  Leak
checking is off: the Python interpreter itself keeps allocations alive at
exit.  (A planted one-element overrun in ``de_cache_slots`` is reported as a
heap-buffer-overflow and fails the test.)
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, os.path.join(ROOT, "paper_2607_24434_amd"))

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="no host C++ compiler")


def test_cache_tests_pass_under_asan_and_ubsan():
    import build_sanitized

    lib = build_sanitized.build()
    env = dict(os.environ)
    env.update(DE_LIBRARY=lib, LD_PRELOAD=build_sanitized.runtime_preload(),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:exitcode=86",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=87",
               CUDA_VISIBLE_DEVICES="", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-s", "-p", "no:cacheprovider",
                        "-m", "not gpu", os.path.join(ROOT, "tests", "test_cache.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    print(out[-3000:])
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in r.stdout
