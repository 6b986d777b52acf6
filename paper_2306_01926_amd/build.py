"""Compile libga.so (HIP C++ for gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libga.so")
SOURCES = [os.path.join(HERE, "csrc", "ga_abi.cpp"), os.path.join(HERE, "csrc", "ga_kernels.hip"),
           os.path.join(HERE, "csrc", "ga_lloyd.hip"),
           os.path.join(HERE, "csrc", "ga_noalloc.hip"),
           os.path.join(HERE, "csrc", "ga_block.hip"),
           os.path.join(HERE, "csrc", "ga_merge.hip"),
           os.path.join(HERE, "csrc", "ga_backward.hip")]


def hipcc() -> str:
    return shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


# Device-code flags of every source: packed FP32 instructions off; MFMA results
# in ordinary VGPRs.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-mfma-vgpr-form", "-I", os.path.join(ROOT, "include")]


def build(verbose: bool = False) -> str:
    cmd = [hipcc(), *DEVICE_FLAGS, "-fPIC", "-shared", *SOURCES, "-o", LIB + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + r.stderr[-6000:])
    if verbose:
        print(r.stderr)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
