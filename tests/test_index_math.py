"""Host check of the kernels' integer index arithmetic (no GPU needed).

`index_math.hpp` holds the multiply-high division, the tile orders and the work ranges of the
persistent stream-K contraction, as `__host__ __device__` functions.  The checker program
(tests/index_math_check.cpp) compiles that same header for the CPU and checks FastDiv against
integer division, the tile orders for bijectivity, and simulates ~20k launches of the schedule:
every (tile, layer) unit done once, every finished tile written once, no partial slot written
twice, and each split tile's fixup summing exactly its own partial sums, every layer once.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2206_08720_amd", "csrc")
ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")


def test_index_math_host_check(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None or not os.path.isdir(ROCM_INCLUDE):
        pytest.skip("needs g++ and the ROCm headers")
    exe = str(tmp_path / "index_math_check")
    subprocess.run([cxx, "-O2", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE, "-I", CSRC,
                    os.path.join(ROOT, "tests", "index_math_check.cpp"), "-o", exe], check=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    print(res.stdout)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip().endswith("OK")
