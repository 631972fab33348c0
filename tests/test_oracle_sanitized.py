"""Host sanitizer run of the oracle: the C oracle built with AddressSanitizer
and UndefinedBehaviorSanitizer (-fno-sanitize-recover, so any report fails
the run), loaded in place of the plain build, under the CPU test suite
(everything but the mutant builds, which compile their own copies, and this
file).  An out-of-bounds access, use after free, signed overflow, misaligned
or null access anywhere in the oracle's C code aborts the child process."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    r = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_suite_under_asan_and_ubsan():
    runtime = _asan_runtime()
    if runtime is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    sys.path.insert(0, ROOT)
    from oracle import build
    lib = build.build(sanitize=True)
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report_load8" in syms and "__ubsan_handle" in syms, "not an instrumented build"
    env = dict(os.environ, LTD_ORACLE_LIB=lib, LD_PRELOAD=runtime,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    here = os.path.basename(__file__)
    cmd = [sys.executable, "-m", "pytest", "tests", "-m", "not gpu", "-q", "-x",
           "-p", "no:cacheprovider", "--ignore", "tests/test_oracle_mutants.py",
           "--ignore", f"tests/{here}",
           "--rootdir", ROOT]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=1500)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail
