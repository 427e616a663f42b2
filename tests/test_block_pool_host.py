"""The KV pool's host bookkeeping (csrc/block_pool.h: the free list, the
per-prompt block tables, the index mapping of a commit's copy into the
prefix) under AddressSanitizer and UndefinedBehaviorSanitizer: a host-only
C++ build of the header with randomized prefill / commit / release
sequences checked against its invariants."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_block_pool_under_sanitizers(tmp_path):
    exe = tmp_path / "block_pool_test"
    src = os.path.join(ROOT, "tests", "native", "block_pool_test.cpp")
    inc = os.path.join(ROOT, "paper_2412_10418_amd", "csrc")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", inc, src, "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "block pool: ok" in r.stdout
