"""Where plan_batch_kernel's time goes, phase by phase.

Runs mp_plan_batch on the batched ResNeXt-like workload (1024 traces of 2000
tensors) with the profiling build libmemoplan_phase.so (built beforehand on
the CPU: python -m paper_2203_00448_amd.build --phase-timing), in which
thread 0 of every workgroup stamps the shader clock (clock64) as its trace
enters each phase, and prints the cycles per phase over the 1024 traces as a
Markdown table.  The kernel is otherwise the production one; four traces
share each CU, so a phase's cycles include the time the other three take the
CU's issue slots.

    python -m paper_2203_00448_amd.phase_clock
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import binding
from . import tracegen as tg
from .build import PHASE_LIB_PATH

SLOTS = 8  # stamps per trace (kPhaseSlots)
PHASES = [
    ("ingest (sizes, first, last into LDS; unit, checks)", 0, 1),
    ("position check (sorted by first; else the position sort)", 1, 2),
    ("reach (band ends)", 2, 3),
    ("prefix (band starts, pair count, live-bytes bound)", 3, 4),
    ("sizes in units, left lists and pending counts, classes", 4, 5),
    ("placement (Kahn rounds)", 5, 6),
    ("output (offsets, peak, bound)", 6, 7),
]


def main() -> None:
    binding._lib = None
    L = binding.load_library(PHASE_LIB_PATH)
    L.mp_debug_phase_clock.argtypes = [ctypes.c_void_p, ctypes.c_int64]
    L.mp_debug_phase_clock.restype = ctypes.c_int32
    n_traces, n = 1024, 2000
    b = tg.resnext_batch(n_traces, n)
    dev = lambda a, t: torch.from_numpy(np.ascontiguousarray(a)).to("cuda", dtype=t)
    args = (dev(b.begin, torch.int64), dev(b.num_ops, torch.int32), dev(b.size, torch.int64),
            dev(b.first, torch.int32), dev(b.last, torch.int32))
    for _ in range(3):  # the stamps of the last call are read
        binding.plan_batch(*args, max_trace_len=n)
    torch.cuda.synchronize()
    buf = (ctypes.c_longlong * (4096 * SLOTS))()
    if L.mp_debug_phase_clock(buf, 4096 * SLOTS) != binding.MP_OK:
        raise RuntimeError("mp_debug_phase_clock failed")
    a = np.frombuffer(buf, dtype=np.int64).reshape(4096, SLOTS)[:n_traces].astype(np.float64)
    total = a[:, 7] - a[:, 0]
    print(f"plan_batch_kernel, {n_traces} traces x {n} tensors, four traces a CU: "
          "shader-clock cycles per trace")
    print()
    print("| phase | mean | max | share of the mean total |")
    print("|---|---|---|---|")
    for name, s0, s1 in PHASES:
        d = a[:, s1] - a[:, s0]
        print(f"| {name} | {d.mean():,.0f} | {d.max():,.0f} | {d.mean() / total.mean():.1%} |")
    print(f"| whole trace | {total.mean():,.0f} | {total.max():,.0f} | 100.0% |")
    q = np.arange(n_traces) // (n_traces // 4)
    print()
    print("whole-trace mean by dispatch quarter (blockIdx / 256):",
          ", ".join(f"{total[q == k].mean():,.0f}" for k in range(4)))


if __name__ == "__main__":
    main()
