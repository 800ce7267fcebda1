"""Build liboscar.so (HIP, gfx950) in-tree with hipcc.

Each translation unit is compiled to an object under _build/ and linked into
paper_2605_17757_amd/liboscar.so.  The cache-update kernel is compiled without
floating-point contraction so that its fp32 steps are single IEEE operations.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "liboscar.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-fno-gpu-flush-denormals-to-zero",
    # no packed fp32 instructions anywhere in this library
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]
SOURCES = {
    "oscar_host.hip": [],
    "append.hip": ["-ffp-contract=off"],
    "decode.hip": [],
    # keep MFMA accumulators in VGPRs: the kernel shifts and reads them with VALU ops
    "decode_mfma.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    # the two-chunk split instances: the same flags and the max-ilp scheduler
    "decode_mfma_wide2.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1", "-mllvm",
                              "-amdgpu-sched-strategy=max-ilp"],
    "bf16_decode.hip": [],
    "mixed.hip": [],
    "calib.hip": ["-ffp-contract=off"],
    "probe.hip": [],
}


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    for src, extra in SOURCES.items():
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        cmd = [HIPCC, *COMMON, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
