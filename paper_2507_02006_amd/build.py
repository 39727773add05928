"""Builds libaires.so (gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libaires.so")
SOURCES = [os.path.join(HERE, "csrc", n) for n in ("aires.cpp", "kernels.hip", "spmm.hip", "normalize.hip", "scratch.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
    # packed fp32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def build(force: bool = True) -> str:
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp%d" % os.getpid()
        subprocess.check_call([HIPCC, *FLAGS, "-o", tmp, *SOURCES])
        os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
