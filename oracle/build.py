"""Builds the CPU oracle (test infrastructure) into oracle/liboracle.so.

Plain g++, one thread, IEEE arithmetic: no fast-math and no FMA contraction,
so each written fp32/fp64 operation is rounded once.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "eprop_oracle.cpp")
LIB = os.path.join(HERE, "liboracle.so")

CXXFLAGS = ["-O2", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
            "-Wall", "-Wextra"]


def build(src: str = SRC, out: str = LIB, extra=()) -> str:
    tmp = out + ".tmp"
    cmd = ["g++", *CXXFLAGS, *extra, src, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(*sys.argv[1:2]))
