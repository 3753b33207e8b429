"""The host code of the library under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

Builds libbitsmoe_san.so (``paper_2606_00079_amd.build --sanitize``: every
.cpp and the host side of every .hip instrumented, device code as usual) and
runs the C-ABI tests against it (argument checking of every entry point,
the host ILP against the oracle's dynamic program and exhaustive search,
layouts and budgets) in a child process that preloads the sanitizer runtime.  Any report (heap overflow, use after
free, undefined behaviour) aborts the child and fails this test.  The
full-size ILP cases are left to the plain build (the instrumented DP is an
order of magnitude slower).
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.slow
def test_host_code_under_asan_ubsan():
    from paper_2606_00079_amd import build as b
    try:
        rt = b.asan_runtime()
    except FileNotFoundError as e:  # pragma: no cover
        pytest.skip(str(e))
    lib = b.build(sanitize=True)
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, BITSMOE_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", "-k", "not full_size",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=900)
    tail = "\n".join(r.stdout.splitlines()[-30:])
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in r.stdout and "runtime error:" not in r.stdout, tail
