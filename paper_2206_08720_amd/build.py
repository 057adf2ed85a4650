"""Build the HIP library libntk.so in-tree for gfx950 (hipcc cross-compiles without a GPU).

    python -m paper_2206_08720_amd.build        # or: from paper_2206_08720_amd.build import build

Every .hip source under csrc/ is compiled to an object in csrc/_build/ (in
parallel), then linked into paper_2206_08720_amd/libntk.so.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(CSRC, "_build")
LIB = os.path.join(PKG, "libntk.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed-fp32 VALU forms are disabled for device code; hipcc's host pass warns that it does
# not know the feature, which is harmless.
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wno-unused-result", "-I", os.path.join(PKG, "..", "include")]
# Per-file extras.  Keep MFMA accumulators in the VGPR form: in diag.hip so that the fp64
# chains are not copied between accumulation and architectural registers every iteration.
PER_FILE = {"diag.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
            # the inside-out kernel feeds an MFMA's result to the next MFMA as an A operand
            "kernels_pairsum.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
            # the fp64 convolution forward otherwise moves its accumulators between the two
            # register files at every group of K tiles
            "kernels_conv.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines()
                    if "packed-fp32-ops" not in l)  # drop the harmless host-pass warning
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose=False, extra_flags=()):
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    if not srcs:
        raise RuntimeError("no HIP sources found")

    def compile_one(src):
        obj = os.path.join(BUILD, os.path.basename(src) + ".o")
        per = PER_FILE.get(os.path.basename(src), [])
        out = _run([HIPCC, *COMMON, *per, *extra_flags, "-c", src, "-o", obj])
        if verbose and out.strip():
            print(out)
        return obj

    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(compile_one, srcs))
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
