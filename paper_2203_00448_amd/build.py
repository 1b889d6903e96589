"""Build libmemoplan.so (HIP for gfx950) in-tree with hipcc, and beside it
libmemoplan_dbgwait.so: the same sources with MP_DEBUG_WAIT, a test build
whose single-trace planner takes its rarely reached late-predecessor paths on
request (MEMOPLAN_DEBUG_WAIT).  The two compile in parallel."""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(PKG, "libmemoplan.so")
DBG_WAIT_LIB_PATH = os.path.join(PKG, "libmemoplan_dbgwait.so")
# profiling build: plan_batch_kernel stamps the clock at each phase of every
# trace (MP_PHASE_TIMING; read by paper_2203_00448_amd.phase_clock).  Built
# only on request: python -m paper_2203_00448_amd.build --phase-timing
PHASE_LIB_PATH = os.path.join(PKG, "libmemoplan_phase.so")

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    # packed-FP32 instructions stay off (no floating point here anyway)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(verbose: bool = False, phase_timing: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    jobs = []
    variants = [(LIB_PATH, []), (DBG_WAIT_LIB_PATH, ["-DMP_DEBUG_WAIT"])]
    if phase_timing:
        variants = [(PHASE_LIB_PATH, ["-DMP_PHASE_TIMING"])]
    for out, extra in variants:
        cmd = [hipcc, *HIPCC_FLAGS, *extra, "-I", INCLUDE, "-I", CSRC, "-o", out + ".tmp",
               *sources()]
        if verbose:
            print(" ".join(cmd), file=sys.stderr)
        jobs.append((out, subprocess.Popen(cmd)))
    failed = [out for out, p in jobs if p.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, f"hipcc ({', '.join(map(os.path.basename, failed))})")
    for out, _ in jobs:
        os.replace(out + ".tmp", out)
    return PHASE_LIB_PATH if phase_timing else LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True, phase_timing="--phase-timing" in sys.argv[1:]))
