"""Build libepic.so (HIP, gfx950) in-tree."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libepic.so")
SOURCES = [os.path.join(CSRC, "epic.hip"), os.path.join(CSRC, "tables.cpp")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def command(out: str) -> list:
    return [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-o", out] + SOURCES


def build_library() -> str:
    tmp = LIB + ".tmp"
    subprocess.check_call(command(tmp))
    os.replace(tmp, LIB)
    return LIB
