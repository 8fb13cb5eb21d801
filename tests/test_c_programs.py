"""The C-level tests of libckpt (tests/c/): programs that call the ABI from
plain C, with no Python or torch in the process, so the library runs on the
HIP runtime it was linked against.

plan_fuzz_san runs here (host code only, under AddressSanitizer and
UndefinedBehaviorSanitizer); abi_roundtrip and its sanitized twin need a GPU.
The programs are built by __graft_entry__.build(); a missing one is built
first.
"""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
C_DIR = os.path.join(HERE, "c")
sys.path.insert(0, C_DIR)
import build_c_tests  # noqa: E402

ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def program(path):
    if not os.path.exists(path):
        build_c_tests.build()
    return path


def run(path, timeout):
    r = subprocess.run([program(path)], capture_output=True, text=True, timeout=timeout, env=ENV)
    sys.stdout.write(r.stdout)
    sys.stderr.write(r.stderr)
    return r


def test_plan_fuzz_sanitized():
    r = run(build_c_tests.PLAN_FUZZ, 300)
    assert r.returncode == 0 and "OK plan_fuzz" in r.stdout


@pytest.mark.gpu
@pytest.mark.parametrize("path", [build_c_tests.ROUNDTRIP, build_c_tests.ROUNDTRIP_SAN],
                         ids=["plain", "sanitized"])
def test_abi_roundtrip_from_c(path):
    r = run(path, 120)
    assert r.returncode == 0 and "OK abi_roundtrip" in r.stdout, r.stderr[-2000:]
