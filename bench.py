#!/usr/bin/env python3
"""Throughput of the static memory-planning hot path on one MI355X.

Workload: the batched ResNeXt-101-like traces -- 1024 independent traces of
2000 tensors each (2,048,000 tensors), seeds [2, b] -- resident in HBM before
timing.  One step plans every trace with greedy-by-size (lowest fitting gap),
computes each trace's live-bytes lower bound, and validates the produced plan
(every lifetime-intersecting pair checked for address overlap; the step
requires zero conflicts).

Prints one JSON line: tensors planned per second, the roofline of the
dominant kernel (the batched planner) from HIP events on its stream beside
the box's measured copy bandwidth, and the plain CPU oracle timed on the
host's cores as a baseline.  After the timed steps, `configs` reports every
workload of the benchmark (outside `value`): the 256-tensor chain (batched
and single-trace planners), the batch itself, the seq2seq-decode-like trace
(100,000 tensors) and the ranking-like trace (1,000,000 tensors) on the
whole-device planner, and the validation and liveness kernels on the decode
trace's plan and a corrupted copy of it -- each with tensors per second,
planned peak over the live-bytes lower bound, a parity flag against the
oracle's digests (tests/golden/expected.json, written by the oracle only),
the dependency depth and the largest degree (tests/golden/workload_stats.json).
A strategies leg compares greedy-by-size, Greedy by Breadth, bump allocation
and the exact optimum on tiny traces.
"""
from __future__ import annotations

import argparse
import hashlib
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
                    help="skip the per-config legs other than the batch (profiling runs)")
    ap.add_argument("--no-strategies", action="store_true",
                    help="skip the strategy-comparison leg")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, copy 256 MiB device to device three times "
                         "(a kernel of known traffic for scaling HBM counters)")
    return ap.parse_args()


def _golden(name):
    with open(os.path.join(ROOT, "tests", "golden", name)) as fh:
        return json.load(fh)["configs"]


def _sha(a):
    import numpy as np
    return hashlib.sha256(np.ascontiguousarray(a).astype("<i8").tobytes()).hexdigest()


def measured_traffic():
    """HBM bytes per launch of the planner kernel from the committed counter
    summary, when it was taken on the current kernel source; else None."""
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


def _timed(torch, np, fn, reps, stream=None):
    """One warm-up call, then `reps` calls each bracketed by HIP events on the
    stream; returns (last result, median ms, min ms)."""
    s = stream if stream is not None else torch.cuda.current_stream()
    fn()
    ms, res = [], None
    for _ in range(reps):
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        ev[0].record(s)
        res = fn()
        ev[1].record(s)
        torch.cuda.synchronize()
        ms.append(ev[0].elapsed_time(ev[1]))
    return res, float(np.median(ms)), float(np.min(ms))


def copy_bandwidth(torch, np, mib: int = 1024, reps: int = 10):
    """Device-to-device copy of `mib` MiB: read + write bytes over the median
    time (the box's practical HBM rate, beside the 8 TB/s peak)."""
    src = torch.empty(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    _, med, _ = _timed(torch, np, lambda: dst.copy_(src), reps)
    del src, dst
    return 2 * (mib << 20) / (med * 1e-3) / 1e9


def _trace_dev(torch, np, t):
    d = lambda a, ty: torch.from_numpy(np.ascontiguousarray(a)).to("cuda", dtype=ty)
    return d(t.size, torch.int64), d(t.first, torch.int32), d(t.last, torch.int32)


def chain256_leg(binding, tg, np, torch, exp, stats, reps=50):
    """The 256-tensor chain: one trace through the batched planner (one
    workgroup) and through the whole-device planner; latency per call."""
    t = tg.chain256()
    b = tg.concat([t])
    d = lambda a, ty: torch.from_numpy(np.ascontiguousarray(a)).to("cuda", dtype=ty)
    bargs = (d(b.begin, torch.int64), d(b.num_ops, torch.int32), d(b.size, torch.int64),
             d(b.first, torch.int32), d(b.last, torch.int32))
    status = binding.new_status()
    (boff, bpeak, blb), bmed, bmin = _timed(
        torch, np, lambda: binding.plan_batch(*bargs, max_trace_len=t.n, check=False,
                                              status=status), reps)
    targs = _trace_dev(torch, np, t)
    (toff, tpeak), tmed, tmin = _timed(
        torch, np, lambda: binding.plan_trace(*targs, t.num_ops, check=False, status=status), reps)
    if int(status.item()) != binding.MP_OK:
        raise SystemExit("chain256: device status " + str(int(status.item())))
    e = exp["chain256"]
    return {"workload": "chain256: 256 tensors, first = i, last = i + 1 + Geometric(0.5), "
                        "sizes 2^U[10,22) rounded to 64 B (seed 1)",
            "tensors": t.n,
            "plan_batch": {"tensors_per_s": t.n / (bmed * 1e-3), "us": bmed * 1e3,
                           "min_us": bmin * 1e3, "calls": reps,
                           "parity": _sha(boff.cpu().numpy()) == e["offsets_sha256"]
                           and int(bpeak.item()) == e["peak"]},
            "plan_trace": {"tensors_per_s": t.n / (tmed * 1e-3), "us": tmed * 1e3,
                           "min_us": tmin * 1e3, "calls": reps,
                           "parity": _sha(toff.cpu().numpy()) == e["offsets_sha256"]
                           and int(tpeak.item()) == e["peak"]},
            "peak": int(tpeak.item()), "lb": int(blb.item()),
            "peak_over_lb": int(tpeak.item()) / int(blb.item()),
            "depth": stats["chain256"]["depth"], "max_degree": stats["chain256"]["max_degree"]}


def single_trace_leg(binding, tg, np, torch, name, t, exp, stats, reps):
    """mp_plan_trace on one large trace, inputs resident in HBM: one warm-up
    call, then `reps` calls timed with HIP events on the stream."""
    args = _trace_dev(torch, np, t)
    n = t.n
    stream = torch.cuda.current_stream()
    offset = torch.empty(n, dtype=torch.int64, device="cuda")
    peak = torch.empty(1, dtype=torch.int64, device="cuda")
    ws = torch.empty(binding.workspace_bytes(binding.OP_PLAN_TRACE, n, t.num_ops, 1),
                     dtype=torch.uint8, device="cuda")
    status = binding.new_status()
    _, med, mn = _timed(torch, np, lambda: binding.plan_trace(
        *args, t.num_ops, check=False, out=(offset, peak), status=status, workspace=ws,
        stream=stream), reps, stream)
    st = int(status.item())
    if st != binding.MP_OK:
        raise SystemExit(f"{name}: device status {st}: {binding.status_string(st)}")
    _, max_live = binding.live_bytes_profile(*args, t.num_ops)
    off = offset.cpu().numpy()
    e = exp[name]
    row = {"tensors": n, "tensors_per_s": n / (med * 1e-3), "ms": med, "min_ms": mn,
           "calls": reps, "peak": int(peak.item()), "lb": int(max_live.item()),
           "peak_over_lb": int(peak.item()) / int(max_live.item()),
           "parity": _sha(off) == e["offsets_sha256"] and int(peak.item()) == e["peak"],
           "depth": stats[name]["depth"], "max_degree": stats[name]["max_degree"],
           "pairs": stats[name]["pairs"]}
    return row, args, offset


def probe_leg(binding, np, torch, t, args, offset, reps=3):
    """The decode plan applied to a slab of its peak and probed by replaying the
    ops (one wave per 256-byte tile)."""
    n = t.n
    peak = int((offset + args[0]).max().item())
    slab = torch.empty(peak, dtype=torch.uint8, device="cuda")
    pws = torch.empty(binding.workspace_size(binding.OP_PROBE, n, t.num_ops), dtype=torch.uint8,
                      device="cuda")
    clob = torch.empty(n, dtype=torch.uint8, device="cuda")
    n_clob = torch.empty(1, dtype=torch.int64, device="cuda")
    status = binding.new_status()
    _, med, _ = _timed(torch, np, lambda: binding.probe_plan(
        *args, offset, t.num_ops, slab, check=False, out=(clob, n_clob), status=status,
        workspace=pws), reps)
    if int(status.item()) != binding.MP_OK or int(n_clob.item()) != 0:
        raise SystemExit("decode100k: the probe of the plan found clobbered tensors")
    probe_bytes = 3 * int(t.size.sum()) + 25 * n  # write, check, clear; inputs and flags
    return {"ms": med, "clobbered": 0, "algorithmic_bytes": probe_bytes,
            "gb_per_s": probe_bytes / (med * 1e-3) / 1e9,
            "kernel": "probe_tiles_kernel (one wave per 256-byte slab tile replays its events in "
                      "op order, after a radix sort of (tile, op) keys)"}


def cfg5_leg(binding, tg, np, torch, t, args, offset, exp, reps=5):
    """Liveness and validation on the decode trace: the per-op live bytes, the
    clean plan (no pair may be reported) and a copy with 100 seed-chosen
    offsets perturbed (exactly the oracle's 2,633 pairs)."""
    status = binding.new_status()
    live = torch.empty(t.num_ops, dtype=torch.int64, device="cuda")
    mx = torch.empty(1, dtype=torch.int64, device="cuda")
    lws = torch.empty(binding.workspace_size(binding.OP_LIVE_BYTES, t.n, t.num_ops),
                      dtype=torch.uint8, device="cuda")
    _, lmed, _ = _timed(torch, np, lambda: binding.live_bytes_profile(
        *args, t.num_ops, check=False, out=(live, mx), status=status, workspace=lws), reps)
    e3 = exp["decode100k"]
    ev = exp["decode100k_validation"]
    cap = ev["corrupted_conflicts"]
    vws = torch.empty(binding.workspace_size(binding.OP_VALIDATE, t.n, 0, cap), dtype=torch.uint8,
                      device="cuda")
    pairs = torch.empty((cap, 2), dtype=torch.int64, device="cuda")
    cnt = torch.empty(1, dtype=torch.int64, device="cuda")
    val = lambda off, srt=False: binding.validate_plan(*args, off, capacity=cap, check=False,
                                                       status=status, workspace=vws,
                                                       out=(pairs, cnt), assume_sorted=srt)
    _, cmed, _ = _timed(torch, np, lambda: val(offset), reps)
    clean = int(cnt.item())
    # the decode trace is in first order: with the caller's sorted-first hint
    # the unsorted path's sorts are not enqueued at all
    _, hmed, _ = _timed(torch, np, lambda: val(offset, True), reps)
    clean_h = int(cnt.item())
    bad, _ = tg.corrupt_offsets(t.first, t.last, offset.cpu().numpy(), seed=5, k=100)
    bad_d = torch.from_numpy(bad).to("cuda")
    _, bhmed, _ = _timed(torch, np, lambda: val(bad_d, True), reps)
    bad_h = (int(cnt.item()), _sha(pairs.cpu().numpy()))
    _, bmed, _ = _timed(torch, np, lambda: val(bad_d), reps)
    if int(status.item()) != binding.MP_OK:
        raise SystemExit("cfg5: device status " + str(int(status.item())))
    return {"workload": "decode100k's plan from the GPU planner, clean and with 100 offsets "
                        "perturbed (seed 5)",
            "live_bytes_profile": {"us": lmed * 1e3, "tensors_per_s": t.n / (lmed * 1e-3),
                                   "ops": t.num_ops,
                                   "parity": _sha(live.cpu().numpy()) == e3["live_sha256"]
                                   and int(mx.item()) == e3["lb"]},
            "validate_clean": {"us": cmed * 1e3, "tensors_per_s": t.n / (cmed * 1e-3),
                               "conflicts": clean, "parity": clean == 0},
            "validate_corrupted": {"us": bmed * 1e3, "tensors_per_s": t.n / (bmed * 1e-3),
                                   "conflicts": int(cnt.item()),
                                   "parity": int(cnt.item()) == cap
                                   and _sha(pairs.cpu().numpy()) == ev["pairs_sha256"]},
            "validate_sorted_hint": {"clean_us": hmed * 1e3, "corrupted_us": bhmed * 1e3,
                                     "parity": clean_h == 0 and bad_h[0] == cap
                                     and bad_h[1] == ev["pairs_sha256"]}}


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
    (_, opt), opt_ms, _ = _timed(torch, np, lambda: binding.optimal_batch(*args), reps)
    low, best, bump, breadth, opt, lb = (x.cpu().numpy().astype(np.float64)
                                         for x in (low, best, bump, breadth, opt, lb))

    def ratio(x):
        r = x / opt
        return {"mean": float(r.mean()), "max": float(r.max()),
                "at_optimum": float((x == opt).mean())}
    return {"workload": f"tiny_batch: {n_traces} ResNeXt-like traces x {n} tensors "
                        "(seeds [6,b]), exact optimum by exhaustive search",
            "optimal_ms": opt_ms, "calls": reps,
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
    (_, breadth), breadth_ms, _ = _timed(torch, np, lambda: binding.plan_breadth_batch(*margs),
                                         reps)
    (_, bump), bump_ms, _ = _timed(
        torch, np, lambda: binding.bump_plan(margs[2], margs[3], margs[4],
                                             int(mbatch.num_ops.max()), begin=margs[0]), reps)
    size_peak, breadth, bump, lb = (x.cpu().numpy().astype(np.float64)
                                    for x in (size_peak, breadth, bump, lb))
    over = lambda x: {"mean": float((x / lb).mean()), "max": float((x / lb).max()),
                      "at_lb": float((x == lb).mean())}
    return {"greedy_size_over_lb": over(size_peak), "greedy_breadth_over_lb": over(breadth),
            "bump_over_lb": over(bump), "breadth_ms": breadth_ms, "bump_ms": bump_ms,
            "breadth_beats_size": float((breadth < size_peak).mean())}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(tg, np, batch, with_single: bool):
    """The plain single-threaded C oracle on the host: the batch on N threads
    (each planning a disjoint set of traces; the calls release the GIL) and on
    one, the chain, the decode trace once, and a prefix of the ranking trace
    (its full run takes minutes).  About 20-30 s of host work in all."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor

    n = int(batch.size.shape[0])
    B = batch.n_traces
    sl = lambda b: slice(int(batch.begin[b]), int(batch.begin[b + 1]))

    def plan_traces(bs):
        for b in bs:
            s = sl(b)
            oracle.plan_trace(batch.size[s], batch.first[s], batch.last[s], int(batch.num_ops[b]))

    threads = max(1, min(os.cpu_count() or 1, int(os.environ.get("OMP_NUM_THREADS", "1024"))))
    parts = [list(range(k, B, threads)) for k in range(threads)]
    passes, dt = 0, 0.0
    with ThreadPoolExecutor(threads) as ex:
        while passes == 0 or dt < 3.0:
            t0 = time.perf_counter()
            list(ex.map(plan_traces, parts))
            dt += time.perf_counter() - t0
            passes += 1
    out = {"value": passes * n / dt, "unit": "tensors/s", "cores": threads, "kind": "oracle",
           "sample": f"{passes} passes over all {B} traces of the batch ({n} tensors each pass), "
                     f"{threads} threads each running the single-threaded oracle on disjoint "
                     "traces",
           "seconds": dt, "cpu_model": cpu_model(), "host_cpus": os.cpu_count()}
    p1, d1 = 0, 0.0
    while p1 == 0 or d1 < 4.0:
        t0 = time.perf_counter()
        plan_traces(range(B))
        d1 += time.perf_counter() - t0
        p1 += 1
    out["single_core"] = {"value": p1 * n / d1, "cores": 1, "seconds": d1,
                          "sample": f"{p1} passes over all {B} traces, one thread"}
    if with_single:
        per = {}
        t = tg.chain256()
        t0 = time.perf_counter()
        for _ in range(20):
            oracle.plan_trace(t.size, t.first, t.last, t.num_ops)
        per["chain256"] = {"tensors_per_s": 20 * t.n / (time.perf_counter() - t0), "cores": 1,
                           "sample": "20 calls"}
        t = tg.decode100k()
        t0 = time.perf_counter()
        oracle.plan_trace(t.size, t.first, t.last, t.num_ops)
        dd = time.perf_counter() - t0
        per["decode100k"] = {"tensors_per_s": t.n / dd, "seconds": dd, "cores": 1,
                             "sample": "one call on the whole trace"}
        t = tg.ranking1m()
        m = 15000
        t0 = time.perf_counter()
        oracle.plan_trace(t.size[:m], t.first[:m], t.last[:m], int(t.last[:m].max()) + 1)
        dd = time.perf_counter() - t0
        per["ranking1m"] = {"tensors_per_s": m / dd, "seconds": dd, "cores": 1,
                            "sample": f"the first {m} tensors ({m // 10} ops; the live set is "
                                      "still growing there, so the whole trace runs slower "
                                      "per tensor)"}
        out["per_config"] = per
    return out


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
    exp, stats = _golden("expected.json"), _golden("workload_stats.json")
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
    e2 = exp["resnext_batch"]
    parity2 = (_sha(offset.cpu().numpy()) == e2["offsets_sha256"]
               and _sha(peak_np) == e2["peaks_sha256"] and _sha(lb_np) == e2["lbs_sha256"])
    copy_gbs = copy_bandwidth(torch, np)

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
        "dtype_note": "offsets int64 in bytes; the planner computes in u32 counts of the common "
                      "power-of-two unit when a trace's sizes sum below 2^31 units (every trace "
                      "here), in 64-bit counts otherwise",
        "data": "synthetic",
        "config": {"workload": "resnext_batch: 1024 ResNeXt-101-like traces x 2000 tensors "
                               "(seeds [2,b]), greedy-by-size lowest fit",
                   "n_traces": n_traces, "tensors": n, "policy": "lowest_fit"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(),
                     "kernel": "plan_batch_kernel", "kernel_avg_us": kern_avg_ms * 1e3,
                     "kernel_min_us": float(np.min(kern_ms)) * 1e3,
                     "algorithmic_bytes": algo_bytes, "copy_gbs": copy_gbs,
                     "frac_of_copy": achieved / copy_gbs},
        "peak_over_lb": {"mean": float(ratio.mean()), "max": float(ratio.max())},
        "validate_us": float(np.mean(val_ms)) * 1e3,
        "conflicts": int(n_conf.item()),
    }
    s2 = stats["resnext_batch"]
    configs = {"cfg2_resnext_batch": {
        "tensors": n, "tensors_per_s": out["value"], "plan_us": kern_avg_ms * 1e3,
        "plan_tensors_per_s": n / (kern_avg_ms * 1e-3), "validate_us": out["validate_us"],
        "peak_over_lb": out["peak_over_lb"], "parity": parity2, "depth": s2["depth"],
        "max_degree": s2["max_degree"], "pairs_per_trace_mean": s2["pairs_per_trace_mean"]}}
    if args.copy_calibration:
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = 2 * src.numel()
    if not args.no_single_trace:
        configs["cfg1_chain256"] = chain256_leg(binding, tg, np, torch, exp, stats)
        t3 = tg.decode100k()
        row3, args3, off3 = single_trace_leg(binding, tg, np, torch, "decode100k", t3, exp, stats,
                                             reps=3)
        row3["workload"] = ("decode100k: 100,000 tensors, 4000 ops x 25 births, Geometric(0.3) "
                            "lifetimes, 2% to the end, Pareto(1.5) sizes (seed 3), lowest fit")
        row3["probe"] = probe_leg(binding, np, torch, t3, args3, off3)
        configs["cfg3_decode100k"] = row3
        configs["cfg5_validation_liveness"] = cfg5_leg(binding, tg, np, torch, t3, args3, off3, exp)
        del args3, off3
        t4 = tg.ranking1m()
        row4, _, _ = single_trace_leg(binding, tg, np, torch, "ranking1m", t4, exp, stats, reps=3)
        row4["workload"] = ("ranking1m: 1,000,000 tensors, 100,000 ops x 10 births, lifetimes "
                            "U(1,1000) ops, sizes log-uniform [64 B, 64 KiB] (seed 4), lowest fit")
        configs["cfg4_ranking1m"] = row4
    out["configs"] = configs
    if not args.no_strategies:
        out["strategies"] = strategies_leg(binding, tg, np, torch,
                                           (batch, (begin, num_ops, size, first, last)))
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(tg, np, batch, not args.no_single_trace)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
