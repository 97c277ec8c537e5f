"""Build libepic.so (HIP, gfx950) in-tree.

The kernels of each item width are a compilation unit of their own
(csrc/epic_w<W>.hip); the units compile in parallel, then link with the C ABI
unit (csrc/epic.hip) and the host tables (csrc/tables.cpp)."""
from __future__ import annotations

import os
import shutil
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libepic.so")
WIDTHS = (1, 2, 4, 8, 16)
SOURCES = ([os.path.join(CSRC, "epic.hip"), os.path.join(CSRC, "tables.cpp")]
           + [os.path.join(CSRC, f"epic_w{w}.hip") for w in WIDTHS])
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build_library() -> str:
    tmp = tempfile.mkdtemp(prefix="epic_build_")
    try:
        objs, procs = [], []
        for src in SOURCES:
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            objs.append(obj)
            procs.append((src, subprocess.Popen([HIPCC] + FLAGS + ["-c", "-o", obj, src])))
        failed = [src for src, p in procs if p.wait() != 0]
        if failed:
            raise RuntimeError("hipcc failed on " + ", ".join(failed))
        out = LIB + ".tmp"
        subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-o", out] + objs)
        os.replace(out, LIB)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return LIB
