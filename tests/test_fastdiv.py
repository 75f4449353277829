"""The kernels' division by a divisor fixed for a launch (csrc/common.h:
make_fastdiv / fdiv), checked on the host against exact integer division.

The same header the kernels include is compiled for the host with hipcc and
run over some 5.6 million (dividend, divisor) pairs: every small dividend,
the largest ones below 2^31, random ones and multiples of the divisor plus
small remainders, for divisors from 1 to 2^31 - 1 (the workloads' extents
among them).  The identity is exact by construction (the magic number's
error term stays below 1/d); this pins the code that implements it.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_fastdiv_matches_integer_division():
    src = os.path.join(ROOT, "tests", "fastdiv", "check_fastdiv.cpp")
    with tempfile.TemporaryDirectory() as tmp:
        exe = os.path.join(tmp, "check_fastdiv")
        cmd = [HIPCC, "-O2", "-std=c++17", "-x", "hip", "--offload-arch=gfx950",
               "-I", os.path.join(ROOT, "paper_2105_13480_amd", "csrc"), src, "-o", exe]
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-4000:]
        run = subprocess.run([exe], capture_output=True, text=True, timeout=120)
        assert run.returncode == 0, run.stdout + run.stderr
        assert "bad 0" in run.stdout, run.stdout
