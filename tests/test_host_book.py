"""CPU tests of the host bookkeeping of the C ABI (csrc/host_book.cpp): the
paged allocator (lowest free block first, all-or-nothing), window validation,
row plans with lag rows and tree masks, commit validation, tree-compaction
moves and the commit itself, plus random steps that check the pools stay
partitioned.  The C++ test (tests/host/host_book_test.cpp) is built with
g++ under AddressSanitizer and UndefinedBehaviorSanitizer; no GPU is used.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_12243_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_book_under_sanitizers(tmp_path):
    exe = tmp_path / "host_book_test"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "host", "host_book_test.cpp"), os.path.join(CSRC, "host_book.cpp"),
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and "ALL OK" in r.stdout, r.stdout + r.stderr
