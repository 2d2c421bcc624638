"""The kernels' payload-range arithmetic (paper_2608_09291_amd/csrc/us_range.h),
compiled for the host and exercised on offsets no valid encoding produces:
decreasing offsets, offsets past the end of the payload, arbitrary words.
For any input the staged range must stay inside the payload (the buffer
descriptor built from it then cannot address memory outside the payload
allocation); for the offsets of a valid encoding it must cover the run's
values and the last window's overhang."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("flags", [["-O2"], ["-O1", "-fsanitize=undefined", "-fno-sanitize-recover=all"]])
def test_payload_range_is_safe(flags):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    tmp = tempfile.mkdtemp(prefix="us_range_")
    exe = os.path.join(tmp, "range_check")
    r = subprocess.run(["g++", "-std=c++17", *flags, "-I", os.path.join(ROOT, "paper_2608_09291_amd", "csrc"),
                        os.path.join(ROOT, "tests", "range_check.cpp"), "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
