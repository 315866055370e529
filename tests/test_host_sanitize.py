"""The engine's host-only C++ (weight-image layout, tiled packing, KV-blob
header codec: csrc/host_layout.cpp) built on the CPU with AddressSanitizer
and UndefinedBehaviorSanitizer and driven by tests/host_fuzz.cpp: random
valid inputs, byte flips, extreme field values and truncations, stopping at
the first sanitizer report or violated property."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_asan_and_ubsan():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "host_fuzz")
        cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
               "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
               "-I", os.path.join(ROOT, "include"),
               os.path.join(ROOT, "tests", "host_fuzz.cpp"),
               os.path.join(ROOT, "paper_2502_15524_amd", "csrc", "host_layout.cpp"), "-o", exe]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                   UBSAN_OPTIONS="print_stacktrace=1")
        r = subprocess.run([exe, "200000"], capture_output=True, text=True, env=env, timeout=600)
        assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
        assert "ok 200000 cases" in r.stdout
