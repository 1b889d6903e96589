#!/usr/bin/env python3
"""Throughput of the static memory-planning hot path on one MI355X.

Workload: the batched ResNeXt-101-like traces -- 1024 independent traces of
2000 tensors each (2,048,000 tensors), seeds [2, b] -- resident in HBM before
timing.  One step plans every trace with greedy-by-size (lowest fitting gap),
computes each trace's live-bytes lower bound, and validates the produced plan
(every lifetime-intersecting pair checked for address overlap; the step
requires zero conflicts).

Prints one JSON line: tensors planned per second, the roofline of the
dominant kernel (the batched planner) from HIP events on its stream, and the
plain CPU oracle timed on the host as a baseline.  After the timed steps, a
single-trace leg plans the seq2seq-decode-like trace (100,000 tensors, 4000
ops, seed 3) with the whole-device planner and reports its tensors per
second and peak / live-bytes lower bound, then applies the plan to a slab
and probes it by replaying the ops; a strategies leg compares, on 2048 tiny
ResNeXt-like traces of 10 tensors, the peaks of greedy-by-size (both fits),
Greedy by Breadth and bump allocation with the exact optimum found on the
GPU, and on the benchmark's traces with the live-bytes lower bound (all
outside `value`).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "tensors planned/sec (batched + single-trace); planned peak / live-bytes lower bound"
HBM_PEAK_GBS = 8000.0
BYTES_PER_TENSOR = 24      # read size 8 + first 4 + last 4, write offset 8
BYTES_PER_TRACE = 28       # read begin 8 + num_ops 4, write peak 8 + lb 8


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip timing the CPU oracle (profiling runs)")
    ap.add_argument("--no-single-trace", action="store_true",
                    help="skip the single-trace leg (profiling runs of the batched step)")
    ap.add_argument("--no-strategies", action="store_true",
                    help="skip the strategy-comparison leg")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, copy 256 MiB device to device three times "
                         "(a kernel of known traffic for scaling HBM counters)")
    return ap.parse_args()


def measured_traffic():
    """HBM bytes per launch of the planner kernel from the committed counter
    summary, when it was taken on the current kernel source; else None."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "plan_batch_kernel_resnext_batch_hbm_counters.md")
    src = os.path.join(ROOT, "paper_2203_00448_amd", "csrc", "plan_batch.hip")
    try:
        text = open(path).read()
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines()
                  if line.startswith(("traffic_bytes_per_launch:", "plan_batch_source_sha256:")))
    if fields.get("plan_batch_source_sha256", "").strip() != sha:
        return None
    return int(fields["traffic_bytes_per_launch"])


def single_trace_leg(binding, tg, np, torch, reps: int = 3):
    """mp_plan_trace on the decode-like trace, inputs resident in HBM: one
    warm-up call, then `reps` calls timed with HIP events on the stream."""
    t = tg.decode100k()
    d = lambda a, ty: torch.from_numpy(np.ascontiguousarray(a)).to("cuda", dtype=ty)
    size, first, last = d(t.size, torch.int64), d(t.first, torch.int32), d(t.last, torch.int32)
    n = int(t.size.shape[0])
    stream = torch.cuda.current_stream()
    offset = torch.empty(n, dtype=torch.int64, device="cuda")
    peak = torch.empty(1, dtype=torch.int64, device="cuda")
    ws = torch.empty(binding.workspace_size(binding.OP_PLAN_TRACE, n, t.num_ops),
                     dtype=torch.uint8, device="cuda")
    status = binding.new_status()
    run = lambda: binding.plan_trace(size, first, last, t.num_ops, check=False, out=(offset, peak),
                                     status=status, workspace=ws, stream=stream)
    run()
    ms = []
    for _ in range(reps):
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        ev[0].record(stream)
        run()
        ev[1].record(stream)
        torch.cuda.synchronize()
        ms.append(ev[0].elapsed_time(ev[1]))
    st = int(status.item())
    if st != binding.MP_OK:
        raise SystemExit(f"single trace: device status {st}: {binding.status_string(st)}")
    _, max_live = binding.live_bytes_profile(size, first, last, t.num_ops)
    med = float(np.median(ms))
    # the plan applied to a slab of its peak and probed by replaying the ops
    slab = torch.empty(int(peak.item()), dtype=torch.uint8, device="cuda")
    pws = torch.empty(binding.workspace_size(binding.OP_PROBE, n, t.num_ops), dtype=torch.uint8,
                      device="cuda")
    clob = torch.empty(n, dtype=torch.uint8, device="cuda")
    n_clob = torch.empty(1, dtype=torch.int64, device="cuda")
    probe = lambda: binding.probe_plan(size, first, last, offset, t.num_ops, slab, check=False,
                                       out=(clob, n_clob), status=status, workspace=pws,
                                       stream=stream)
    probe()
    pms = []
    for _ in range(reps):
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        ev[0].record(stream)
        probe()
        ev[1].record(stream)
        torch.cuda.synchronize()
        pms.append(ev[0].elapsed_time(ev[1]))
    if int(status.item()) != binding.MP_OK or int(n_clob.item()) != 0:
        raise SystemExit("single trace: the probe of the plan found clobbered tensors")
    pmed = float(np.median(pms))
    probe_bytes = 3 * int(t.size.sum()) + 25 * n  # write, check, clear; inputs and flags
    return {"workload": "decode100k: 100,000 tensors, 4000 ops x 25 births, Geometric(0.3) "
                        "lifetimes, 2% to the end, Pareto(1.5) sizes (seed 3), lowest fit",
            "tensors_per_s": n / (med * 1e-3), "ms": med, "calls": reps,
            "peak_over_lb": int(peak.item()) / int(max_live.item()),
            "probe": {"ms": pmed, "clobbered": 0, "algorithmic_bytes": probe_bytes,
                      "gb_per_s": probe_bytes / (pmed * 1e-3) / 1e9,
                      "kernel": "probe_tiles_kernel (one wave per 256-byte slab tile replays "
                                "its events in op order, after a radix sort of (tile, op) keys)"}}


def _timed(torch, np, fn, reps):
    fn()  # warm-up
    ms, res = [], None
    for _ in range(reps):
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        ev[0].record()
        res = fn()
        ev[1].record()
        torch.cuda.synchronize()
        ms.append(ev[0].elapsed_time(ev[1]))
    return res, float(np.median(ms))


def strategies_leg(binding, tg, np, torch, medium, n_traces: int = 2048, n: int = 10,
                   reps: int = 3):
    """Peaks of the strategies Sections 2.3 and 6 compare: on tiny traces
    against the optimum of Eq. 2.1 found exactly (mp_optimal_batch), and on the
    benchmark's ResNeXt-like traces against the live-bytes lower bound."""
    batch = tg.tiny_batch(n_traces, n)
    d = lambda a, t: torch.from_numpy(np.ascontiguousarray(a)).to("cuda", dtype=t)
    args = (d(batch.begin, torch.int64), d(batch.num_ops, torch.int32),
            d(batch.size, torch.int64), d(batch.first, torch.int32), d(batch.last, torch.int32))
    _, low, lb = binding.plan_batch(*args, max_trace_len=n)
    _, best, _ = binding.plan_batch(*args, max_trace_len=n, policy=binding.BEST_FIT)
    _, bump = binding.bump_plan(args[2], args[3], args[4], n, begin=args[0])
    _, breadth = binding.plan_breadth_batch(*args)
    binding.optimal_batch(*args)  # warm-up
    ms = []
    for _ in range(reps):
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        ev[0].record()
        off, opt = binding.optimal_batch(*args)
        ev[1].record()
        torch.cuda.synchronize()
        ms.append(ev[0].elapsed_time(ev[1]))
    low, best, bump, breadth, opt, lb = (x.cpu().numpy().astype(np.float64)
                                         for x in (low, best, bump, breadth, opt, lb))

    def ratio(x):
        r = x / opt
        return {"mean": float(r.mean()), "max": float(r.max()),
                "at_optimum": float((x == opt).mean())}
    return {"workload": f"tiny_batch: {n_traces} ResNeXt-like traces x {n} tensors "
                        "(seeds [6,b]), exact optimum by exhaustive search",
            "optimal_ms": float(np.median(ms)), "calls": reps,
            "greedy_lowest_over_opt": ratio(low), "greedy_best_over_opt": ratio(best),
            "breadth_over_opt": ratio(breadth), "bump_over_opt": ratio(bump),
            "opt_over_lb": {"mean": float((opt / lb).mean()), "max": float((opt / lb).max()),
                            "at_lb": float((opt == lb).mean())},
            "resnext_batch": medium_comparison(binding, np, torch, *medium, reps)}


def medium_comparison(binding, np, torch, mbatch, margs, reps):
    """The benchmark's 1024 ResNeXt-like traces of 2000 tensors: each strategy's
    peak over the live-bytes lower bound (the optimum is out of reach)."""
    max_len = int((mbatch.begin[1:] - mbatch.begin[:-1]).max())
    _, size_peak, lb = binding.plan_batch(*margs, max_trace_len=max_len)
    (_, breadth), breadth_ms = _timed(torch, np, lambda: binding.plan_breadth_batch(*margs), reps)
    (_, bump), bump_ms = _timed(
        torch, np, lambda: binding.bump_plan(margs[2], margs[3], margs[4],
                                             int(mbatch.num_ops.max()), begin=margs[0]), reps)
    size_peak, breadth, bump, lb = (x.cpu().numpy().astype(np.float64)
                                    for x in (size_peak, breadth, bump, lb))
    over = lambda x: {"mean": float((x / lb).mean()), "max": float((x / lb).max()),
                      "at_lb": float((x == lb).mean())}
    return {"greedy_size_over_lb": over(size_peak), "greedy_breadth_over_lb": over(breadth),
            "bump_over_lb": over(bump), "breadth_ms": breadth_ms, "bump_ms": bump_ms,
            "breadth_beats_size": float((breadth < size_peak).mean())}


def cpu_baseline(batch, min_seconds: float = 10.0):
    """The plain single-threaded C oracle over the whole batch, repeated until
    about ten seconds of host CPU work, scaled to tensors per second."""
    import oracle
    n = int(batch.size.shape[0])
    passes, dt = 0, 0.0
    while passes == 0 or dt < min_seconds:
        t0 = time.perf_counter()
        oracle.plan_batch(batch.begin, batch.num_ops, batch.size, batch.first, batch.last)
        dt += time.perf_counter() - t0
        passes += 1
    return {"value": passes * n / dt, "unit": "tensors/s", "cores": 1, "kind": "oracle",
            "sample": f"{passes} passes over all {batch.n_traces} traces ({n} tensors each pass), "
                      "single thread",
            "seconds": dt}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2203_00448_amd import binding
    from paper_2203_00448_amd import tracegen as tg

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    binding.load_library()
    batch = tg.resnext_batch(1024, 2000)
    n_traces, n = batch.n_traces, int(batch.size.shape[0])
    d = lambda a, t: torch.from_numpy(np.ascontiguousarray(a)).to("cuda", dtype=t)
    begin, num_ops = d(batch.begin, torch.int64), d(batch.num_ops, torch.int32)
    size, first, last = d(batch.size, torch.int64), d(batch.first, torch.int32), d(batch.last, torch.int32)
    offset = torch.empty(n, dtype=torch.int64, device="cuda")
    peak = torch.empty(n_traces, dtype=torch.int64, device="cuda")
    lb = torch.empty(n_traces, dtype=torch.int64, device="cuda")
    status = binding.new_status()
    stream = torch.cuda.current_stream()
    cap = 1024
    pairs = torch.empty((cap, 2), dtype=torch.int64, device="cuda")
    n_conf = torch.empty(1, dtype=torch.int64, device="cuda")
    vws = torch.empty(binding.workspace_size(binding.OP_VALIDATE_BATCH, n, n_traces, cap),
                      dtype=torch.uint8, device="cuda")

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        binding.plan_batch(begin, num_ops, size, first, last, max_trace_len=2000, check=False,
                           out=(offset, peak, lb), status=status, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        binding.validate_batch(begin, size, first, last, offset, capacity=cap, check=False,
                               status=status, workspace=vws, stream=stream, out=(pairs, n_conf),
                               assume_sorted=True, max_trace_len=2000)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3))
              for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    st = int(status.item())
    if st != binding.MP_OK:
        raise SystemExit(f"device status {st}: {binding.status_string(st)}")
    if int(n_conf.item()) != 0:
        raise SystemExit(f"validation found {int(n_conf.item())} conflicting pairs")

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    kern_ms = [ev[0].elapsed_time(ev[1]) for ev in events]
    val_ms = [ev[1].elapsed_time(ev[2]) for ev in events]
    kern_avg_ms = float(np.mean(kern_ms))
    algo_bytes = BYTES_PER_TENSOR * n + BYTES_PER_TRACE * n_traces
    achieved = algo_bytes / (kern_avg_ms * 1e-3) / 1e9
    peak_np, lb_np = peak.cpu().numpy(), lb.cpu().numpy()
    ratio = peak_np / lb_np

    out = {
        "metric": METRIC,
        "value": n / (ms_per_step * 1e-3),
        "unit": "tensors/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": "resnext_batch: 1024 ResNeXt-101-like traces x 2000 tensors "
                               "(seeds [2,b]), greedy-by-size lowest fit",
                   "n_traces": n_traces, "tensors": n, "policy": "lowest_fit"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(),
                     "kernel": "plan_batch_kernel", "kernel_avg_us": kern_avg_ms * 1e3,
                     "kernel_min_us": float(np.min(kern_ms)) * 1e3,
                     "algorithmic_bytes": algo_bytes},
        "peak_over_lb": {"mean": float(ratio.mean()), "max": float(ratio.max())},
        "validate_us": float(np.mean(val_ms)) * 1e3,
        "conflicts": int(n_conf.item()),
    }
    if args.copy_calibration:
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = 2 * src.numel()
    if not args.no_single_trace:
        out["single_trace"] = single_trace_leg(binding, tg, np, torch)
    if not args.no_strategies:
        out["strategies"] = strategies_leg(binding, tg, np, torch,
                                           (batch, (begin, num_ops, size, first, last)))
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(batch)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
