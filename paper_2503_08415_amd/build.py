"""Build the HIP library of the sweep for gfx950 (in-tree shared object)."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libts_sweep.so")
SOURCES = [os.path.join(CSRC, f) for f in ("host.hip", "sim_kernel.hip", "noalloc.hip")]
HEADERS = [os.path.join(CSRC, f) for f in ("sweep_internal.h", "sweep_host.h")] + [
    os.path.join(INCLUDE, "ts_sweep.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # bit-exact fp64 roofline: no fused multiply-add anywhere
    "-ffp-contract=off",
    # no packed fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # the ILP-first machine scheduler: fewer spills in the 256-slot kernels
    # (about 3 % faster there, no change elsewhere)
    "-mllvm", "-amdgpu-sched-strategy=max-ilp",
    "-Wall", "-Wno-unused-function",
]


def build(verbose: bool = False, out: str = LIB, extra_flags=()) -> str:
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    return out


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(s) > t for s in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
