"""Host check of the reconstruction's one rounding to FP64 (Alg. 3), on the
CPU: the device functions of paper_2609_09095_amd/csrc/fp64_round.hpp are
compiled with g++ (the two HIP function qualifiers and __mul24 supplied as
macros) together with tests/host/rounding_check.cpp, which compares the
FP64 fast path with the 128-bit integer path on random digit vectors and on
values at and next to every rounding boundary, subnormal and overflow
scales and the lift.  The 128-bit path itself is held to the oracle bit for
bit by the GPU parity tests; this test shows the fast path never departs
from it."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_09095_amd", "csrc")
SRC = os.path.join(ROOT, "tests", "host", "rounding_check.cpp")


def test_fast_rounding_never_departs_from_exact(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    exe = str(tmp_path / "rounding_check")
    cmd = [gxx, "-O2", "-std=c++20", "-D__device__=", "-D__forceinline__=inline",
           "-D__mul24(a,b)=((a)*(b))", f"-I{CSRC}", "-o", exe, SRC]
    build = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert build.returncode == 0, build.stderr
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "mismatches 0" in run.stdout
