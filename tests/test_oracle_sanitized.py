"""The oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer
(host code, CPU only): the pin suite runs in a child process against an
ASan/UBSan build of oracle.c, so an out-of-bounds access, a use after free or
undefined behaviour in any pinned path fails the run.  ThreadSanitizer is not
used: the system OpenMP runtime is not instrumented, so every parallel loop
would be reported."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    path = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True,
                          text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.slow
def test_oracle_pins_under_asan_and_ubsan():
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = oracle.build(force=True, sanitize=True)
    env = dict(os.environ)
    env["PLSTM_ORACLE_LIB"] = lib
    env["LD_PRELOAD"] = " ".join(p for p in (asan, env.get("LD_PRELOAD", "")) if p)
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = "4"
    probe = subprocess.run(
        [sys.executable, "-c", "import ctypes, oracle; oracle._load(); "
         "print(oracle._LIB, hasattr(ctypes.CDLL(None), '__asan_init'))"],
        cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert probe.stdout.split() == [lib, "True"], probe.stdout + probe.stderr[-2000:]
    res = subprocess.run(
        [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
         os.path.join(ROOT, "tests", "test_oracle_pins.py"),
         "-k", "not sanitized"],
        cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (res.stdout + res.stderr)[-4000:]
    assert res.returncode == 0, tail
    assert "passed" in res.stdout and "AddressSanitizer" not in res.stderr, tail
    assert "runtime error" not in res.stderr, tail
