"""The host-side bookkeeping under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

The slot table, the KV-block pool and the continuous-batching scheduler
(csrc/host_state.cpp, with the host test surface csrc/host_test_api.cpp) are
built a second time with -fsanitize=address,undefined, and the host tests that
drive them -- the ABI bookkeeping tests, the scheduler tests and the random
call sequences -- run again against that build in a child Python process that
preloads the sanitizer runtimes.  Any invalid access, leak-free use-after-free
or undefined behaviour aborts the child, so the test fails.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST_TESTS = ["tests/test_abi_host.py", "tests/test_serve_host.py", "tests/test_slot_table_property.py"]


@pytest.mark.slow
def test_host_tests_pass_under_asan_and_ubsan():
    from paper_2403_12900_amd import build_host_sanitized as san
    lib = san.build(verbose=False)
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    assert "__asan_report_load" in syms and "__ubsan_handle" in syms, "the library is not instrumented"
    env = dict(os.environ)
    env.update({"LD_PRELOAD": san.runtime_preload(), "SPROUT_HOST_LIB": lib,
                # CPython itself keeps allocations alive at exit; the library's own leaks are not in scope.
                "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1", "UBSAN_OPTIONS": "print_stacktrace=1"})
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", *HOST_TESTS],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert " passed" in r.stdout and "failed" not in r.stdout, tail
