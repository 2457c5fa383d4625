"""The processor-sharing evaluator divides in integers only: ceil_div_small
(kernels.h) takes a reciprocal floor(2^48 / w) from the problem table and
corrects the estimate with one remainder step.  Compiled for the host, it is
checked against exact division for every rate the tables can hold and
dividends at, just below and just above multiples of the rate, up to the
largest work the guards allow (2^46 - 1).  The GPU tests of the sharing
evaluator check the device build against the oracle."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_ceil_div_small_is_exact(tmp_path):
    cc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    cc = cc if os.path.exists(cc) else shutil.which("hipcc")
    if cc is None:
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "arith")
    subprocess.check_call([cc, "-O2", "-std=c++17", "-x", "hip", "--offload-arch=gfx950",
                           "--cuda-host-only", "-I" + os.path.join(ROOT, "include"),
                           "-I" + os.path.join(ROOT, "paper_2607_22242_amd", "csrc"),
                           os.path.join(ROOT, "tests", "host_search", "arith.cpp"), "-o", exe],
                          stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
    bad, checked = map(int, subprocess.run([exe], capture_output=True, text=True,
                                           timeout=120).stdout.split())
    assert checked > 65000 * 20 and bad == 0
