"""The oracle and the C ABI's host paths under AddressSanitizer + UBSan (CPU only).

Builds the host-sanitizer variants of libjetlong and the oracle, then runs the
oracle pins and the ABI tests in a child process that preloads clang's shared
sanitizer runtime and loads those variants.  Any sanitizer report aborts the
child, so the test fails on the first one.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_pins_and_abi_under_asan_ubsan():
    from paper_2607_07740_amd import build_sanitized as bs
    try:
        rt = bs.runtime()
    except FileNotFoundError:
        pytest.skip("clang's shared ASan runtime is not installed")
    lib, oracle_lib = bs.build()
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, JETLONG_LIB=lib, JETLONG_ORACLE_LIB=oracle_lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
           "tests/test_oracle_pins.py", "tests/test_abi.py"]
    res = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
