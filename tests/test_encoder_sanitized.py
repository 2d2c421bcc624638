"""The host encoder and byte accounting under AddressSanitizer and UBSan.

Builds us_encode.cpp (plain C++, host only) together with
tests/sanitize_encode.cpp with g++ and the sanitizers, and runs it: every
encoder mode (4-bit, row-reordered, 2-bit) over sparsities 0 to 1 and padded
leading dimensions, us_pmr, us_pmr_formats, us_iebme_free and the error
paths. Any out-of-bounds access, leak or undefined behaviour fails the test.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_encoder_under_address_and_ub_sanitizers():
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    tmp = tempfile.mkdtemp(prefix="us_san_")
    exe = os.path.join(tmp, "sanitize_encode")
    build = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
             "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "include"),
             os.path.join(ROOT, "tests", "sanitize_encode.cpp"),
             os.path.join(ROOT, "paper_2608_09291_amd", "csrc", "us_encode.cpp"), "-o", exe, "-lpthread"]
    r = subprocess.run(build, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "done, 0 failures" in r.stdout
