"""The host library (planner, block tables, ring map, plan abort, frame
planning, admission) under AddressSanitizer and UndefinedBehaviorSanitizer:
it is built by g++ with the gfx950 launch interface replaced by host
stand-ins, and the host tests run against it in a child process with the
sanitizer runtime preloaded.  Any sanitizer report fails the test.  (The
address-space-limit test of host allocation failures is left out: it cannot
run under the sanitizer's shadow memory.)"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_tests_pass_under_asan_and_ubsan():
    if not shutil.which("g++"):
        pytest.skip("g++ not available")
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    if not asan or not os.path.exists(asan):
        pytest.skip("no AddressSanitizer runtime")
    sys.path.insert(0, ROOT)
    from paper_2607_02640_amd import build
    lib = build.build_host_sanitized()
    env = dict(os.environ, MTN_LIB=lib, LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:allocator_may_return_null=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p",
                        "no:cacheprovider", "-k", "not allocation_failure",
                        "tests/test_abi_host.py", "tests/test_admission.py",
                        "tests/test_index_model_pins.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in out
