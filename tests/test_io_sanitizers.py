"""Host sanitizer runs of the LIBSVM-format IO (paper_2202_12674_amd/csrc/io.cpp).

The driver tests/native/io_sanitize.cpp links io.cpp alone (no GPU code) and
checks bit-exact round trips at several thread counts, edge and malformed
files, and a seeded fuzz of random and mutated files through scan, read and
model read. It is built twice with g++: AddressSanitizer + UndefinedBehavior-
Sanitizer (memory safety of the parser), and ThreadSanitizer (the reader and
writers split files over threads).
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "paper_2202_12674_amd", "csrc", "io.cpp"),
       os.path.join(ROOT, "tests", "native", "io_sanitize.cpp")]
INC = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2202_12674_amd", "csrc")]


def _build_and_run(tmp_path, flags, rounds):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "io_sanitize")
    subprocess.run([gxx, "-std=c++17", "-O1", "-g", *flags, *INC, *SRC, "-o", exe, "-lpthread"],
                   check=True, capture_output=True, timeout=240)
    scratch = tmp_path / "scratch"
    scratch.mkdir()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", TSAN_OPTIONS="halt_on_error=1")
    res = subprocess.run([exe, str(scratch), str(rounds)], capture_output=True, text=True,
                         timeout=300, env=env)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "0 failures" in res.stdout
    return res.stdout


def test_io_under_address_and_undefined_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"],
                         2000)
    assert "models read" in out


def test_io_under_thread_sanitizer(tmp_path):
    _build_and_run(tmp_path, ["-fsanitize=thread"], 300)
