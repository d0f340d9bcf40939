"""The paged-KV host bookkeeping (csrc/kv_pages.h) built on its own with g++ under the
address and undefined-behaviour sanitizers, with bounds-checked standard containers, and
run: allocation, group fork, growth, release and a random operation sequence, each step
followed by the book's consistency check (tests/kv_pages_host_test.cpp)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2505_17218_amd", "csrc")


def test_kv_pages_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "kv_pages_host_test")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-D_GLIBCXX_ASSERTIONS", "-I", CSRC,
           os.path.join(HERE, "kv_pages_host_test.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "kv_pages host test ok" in r.stdout
