"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The library is built with host-side instrumentation (``build.py --sanitize``:
the argument validation, workspace planning and launch sequencing of
api.cpp and the launchers; device code unchanged), and the ABI tests, which
exercise that host code without a GPU, run against it in a child process
with the sanitizer runtime preloaded.  Any sanitizer report fails the test.
There are no float atomics anywhere in the path, so the determinism tests
stand in for a race detector on the device side.
"""
import os
import subprocess
import sys

import pytest

from paper_2609_33614_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_tests_pass_under_asan_and_ubsan(tmp_path):
    try:
        runtime = B.sanitizer_runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    lib = str(tmp_path / "libeat_sanitized.so")
    B.build(jobs=min(8, os.cpu_count() or 1), out=lib, sanitize=True)
    env = dict(os.environ, EAT_LIB_PATH=lib, LD_PRELOAD=runtime,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # -s: a sanitizer writes its report to the process's stderr, which
    # pytest's own capture would swallow when the report ends the process
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"), "-q", "-s",
                        "-p", "no:cacheprovider"], env=env, cwd=ROOT, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert "runtime error:" not in out and "ERROR: AddressSanitizer" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in out, out[-2000:]
