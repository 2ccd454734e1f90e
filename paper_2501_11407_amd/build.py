"""Builds the gfx950 e-prop library in-tree: paper_2501_11407_amd/libeprop.so.

hipcc, one shared object from csrc/kernels.hip (device code) and csrc/eprop.hip
(host side of the C ABI in include/eprop.h).

Flags:
  -ffp-contract=off              no implicit fused multiply-add: the neuron
                                 step rounds each written operation, like the
                                 fp32 spike decisions it must reproduce
  -fno-gpu-flush-denormals-to-zero   IEEE fp32 denormals
  -Xclang -target-feature -Xclang -packed-fp32-ops
                                 no packed fp32 instructions (v_pk_*_f32)
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SOURCES = [os.path.join(PKG, "csrc", "kernels.hip"), os.path.join(PKG, "csrc", "eprop.hip")]
LIB = os.path.join(PKG, "libeprop.so")
ARCH = "gfx950"

HIPFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    return "hipcc"


def build(out: str = LIB, extra=()) -> str:
    tmp = out + ".tmp"
    cmd = [hipcc(), *HIPFLAGS, *extra, "-I", os.path.join(ROOT, "include"), *SOURCES, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(*sys.argv[1:2]))
