"""The host code of libsra (scheduler and C ABI) under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds the host-only library of `build.py --sanitize` (g++, kernel launchers stubbed out) and
runs the schedule and ABI tests against it in a child Python with libasan preloaded: every
schedule the bit-exact tests expand and every validation path of the ABI tests then runs
with bounds, lifetime and undefined-behaviour checks. Any sanitizer report fails the child.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_schedule_and_abi_tests_pass_under_asan_and_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2606_13872_amd import build

    lib = build.build_sanitized()
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(asan):
        pytest.skip("libasan is not installed")
    env = dict(os.environ, SRA_HOST_LIB=lib, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_schedule.py"), os.path.join(ROOT, "tests", "test_abi.py")],
                       capture_output=True, text=True, env=env, cwd=ROOT, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
