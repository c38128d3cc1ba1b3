"""The oracle's pins, run once more against an AddressSanitizer +
UndefinedBehaviorSanitizer build of oracle.c (host code; no GPU).

A child interpreter with the ASan runtime preloaded loads the sanitized
library through SPDP_ORACLE_LIB and runs every tests/test_oracle_*.py pin;
any out-of-bounds access, use after free or undefined behaviour (signed
overflow, bad shift, misaligned access) in the oracle aborts it.
"""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                          check=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.slow
def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc has no AddressSanitizer runtime")
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_asan.so"))
    env = dict(os.environ)
    env.update({
        "SPDP_ORACLE_LIB": lib,
        "LD_PRELOAD": asan,
        # the interpreter itself is not instrumented: leaks of its own are not
        # the oracle's
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "OMP_NUM_THREADS": "4",
    })
    pins = sorted(f for f in os.listdir(os.path.join(ROOT, "tests"))
                  if f.startswith("test_oracle_") and f.endswith(".py"))
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
           *[os.path.join("tests", f) for f in pins]]
    out = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=1500)
    tail = (out.stdout + out.stderr)[-3000:]
    assert out.returncode == 0, tail
    assert "passed" in out.stdout and "AddressSanitizer" not in out.stderr, tail
    assert "runtime error" not in out.stderr, tail
