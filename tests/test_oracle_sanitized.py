"""The oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer.

A copy of oracle/qlayer_oracle.c is built with -fsanitize=address,undefined
(host code only: the oracle is plain C, built with gcc) and the CPU pins of
the oracle run against it in a child process, with the ASan runtime preloaded
into the interpreter.  Any out-of-bounds access, use after free or undefined
behaviour (signed overflow, misaligned access, invalid shift) in the loops the
pins exercise aborts the child, so the test fails.  Leak checking is off: the
interpreter itself keeps memory until exit.
"""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    res = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = res.stdout.strip()
    return path if res.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_pass_under_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    lib = oracle.build(force=True, out=str(tmp_path / "liboracle_san.so"),
                       extra_flags=("-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                                    "-fno-sanitize-recover=all"))
    env = dict(os.environ, ORACLE_LIB=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    files = ["tests/test_oracle_pins.py", "tests/test_oracle_neurons.py", "tests/test_oracle_depthwise.py",
             "tests/test_oracle_epilogue.py"]
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *files],
                         capture_output=True, text=True, cwd=ROOT, env=env, timeout=1500)
    tail = (res.stdout + res.stderr)[-4000:]
    assert res.returncode == 0, tail
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, tail
