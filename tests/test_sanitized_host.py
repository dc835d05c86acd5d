"""The library's host code (argument checks, launch plans, dispatch) under
AddressSanitizer and UndefinedBehaviorSanitizer: a sanitized build runs the
CPU suites that call into it (ABI checks and the bench's host logic).  No
GPU: every call these suites make returns before any HIP launch."""
import os
import subprocess
import sys

import pytest

from paper_2406_18832_amd import build_lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(900)
def test_host_code_under_asan_and_ubsan(tmp_path):
    lib = build_lib.build(sanitize=True, out=str(tmp_path / "libot.so"))
    env = dict(os.environ)
    env.update(LD_PRELOAD=build_lib.asan_runtime(), OT_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    run = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                          "-p", "no:cacheprovider", "tests/test_abi_cpu.py",
                          "tests/test_bench_host.py"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = (run.stdout + run.stderr)[-4000:]
    assert run.returncode == 0, tail
    assert "passed" in run.stdout and "AddressSanitizer" not in run.stderr, tail
    assert "runtime error" not in run.stderr, tail
