"""The host library (allocator, page tables, eviction and decode planning,
every ABI entry point's validation) under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: store.cpp is compiled by g++ with
both, the sanitizer runtimes are preloaded into a fresh interpreter, and the
metadata-only host tests run against that library.  Any report aborts the
run."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

RUNNER = r"""
import sys
import paper_2602_22603_amd.sq as s
s.LIB_PATH = sys.argv[1]
lib = s.lib()
maps = open("/proc/self/maps").read()
assert sys.argv[1] in maps, "the sanitized library is not the one loaded"
assert "libasan" in maps and "libubsan" in maps, "sanitizer runtimes not loaded"
import pytest
sys.exit(pytest.main(["-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                      "tests/test_abi_host.py"]))
"""


@pytest.mark.timeout(900)
def test_host_library_under_asan_and_ubsan(tmp_path):
    from paper_2602_22603_amd import build_lib
    try:
        runtimes = build_lib.sanitizer_runtimes()
    except RuntimeError as err:
        pytest.skip(str(err))
    path = build_lib.build_sanitized(str(tmp_path))
    env = dict(os.environ)
    env["LD_PRELOAD"] = ":".join(runtimes)
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    res = subprocess.run([sys.executable, "-c", RUNNER, path], cwd=ROOT, env=env,
                         capture_output=True, text=True, timeout=800)
    tail = (res.stdout + res.stderr)[-4000:]
    assert res.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
    assert " passed" in res.stdout, tail
