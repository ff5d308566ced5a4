"""Build libturboattn.so (the gfx950 HIP kernels behind the C ABI) in-tree."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libturboattn.so")
SRC = os.path.join(HERE, "csrc", "turbo_api.hip")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # every binary32 operation as written: no FMA contraction
    "-ffp-contract=off",
    # no packed fp32 VALU instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
]
# Translation units and their extra flags.  The attention kernels keep MFMA
# results in VGPRs (no AGPR round trips before the VALU reads them); the
# projection keeps its 256 accumulators per lane in the AGPR file.
UNITS = [
    (os.path.join(HERE, "csrc", "turbo_api.hip"), ["-mllvm", "-amdgpu-mfma-vgpr-form"]),
    (os.path.join(HERE, "csrc", "qkv_project.hip"), []),
]
FLAGS = COMMON  # flags every unit is compiled with


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    objs = []
    for src, extra in UNITS:
        obj = os.path.join(HERE, "_obj_" + os.path.basename(src) + ".o")
        cmd = [HIPCC, *COMMON, *extra, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        objs.append(obj)
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    for obj in objs:
        os.remove(obj)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
