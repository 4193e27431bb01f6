"""Compile libaladdin for gfx950 (in-tree; the built .so travels with the repo)."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libaladdin.so")
SOURCES = [os.path.join(CSRC, f) for f in ("ald_host.cpp", "ald_kernels.hip", "ald_commit.hip", "ald_commit_c.hip", "ald_commit_d.hip",
                                                  "ald_commit_dc.hip",
                                                  "ald_rebalance.hip", "ald_move.hip")]
HEADERS = [os.path.join(CSRC, f) for f in ("ald_internal.h", "ald_device.h", "ald_commit.h", "ald_rebalance.h", "ald_move.h")] + [
    os.path.join(ROOT, "include", "aladdin.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# fp64 results must be single correctly-rounded operations in the written order:
# no contraction into fused multiply-add, no fast-math.  Packed fp32 ops are
# kept out of the generated code.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off",
         "-fno-fast-math", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include")]


def build(verbose: bool = True) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + ["-o", tmp] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


def stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in SOURCES + HEADERS)


if __name__ == "__main__":
    build()
    sys.exit(0)
