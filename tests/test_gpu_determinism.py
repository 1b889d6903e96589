"""Repeatability of every GPU entry point whose kernels run concurrently.

The single-trace planner polls for predecessors placed by other workgroups,
the validation and probe paths count and scatter with device atomics, and
the batched planner appends ready tensors in whatever order its waves reach
the counters.  None of that may change a result: each entry point is called
ten times on the same inputs and every call must equal the oracle's digest
(or the first call, where the result has no stored digest), stopping at the
first mismatch.  Expected digests come from tests/golden/make_expected.py
(oracle only).
"""
import hashlib
import json
import os

import numpy as np
import pytest

from gpu_util import batch_to_device, dev, host, need_gpu, torch
from paper_2203_00448_amd import tracegen as tg

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))
REPEATS = 10


def _expected(name):
    with open(os.path.join(HERE, "golden", "expected.json")) as fh:
        return json.load(fh)["configs"][name]


def _sha(a):
    return hashlib.sha256(np.ascontiguousarray(a).astype("<i8").tobytes()).hexdigest()


def _decode_plan(binding):
    """decode100k planned on the GPU; equal to the oracle's plan by digest."""
    t = tg.decode100k()
    args = (dev(t.size, torch.int64), dev(t.first, torch.int32), dev(t.last, torch.int32))
    off, _ = binding.plan_trace(*args, t.num_ops)
    off = host(off)
    assert _sha(off) == _expected("decode100k")["offsets_sha256"]
    return t, args, off


def test_plan_trace_repeats_decode100k():
    binding = need_gpu()
    t = tg.decode100k()
    exp = _expected("decode100k")
    args = (dev(t.size, torch.int64), dev(t.first, torch.int32), dev(t.last, torch.int32))
    for k in range(REPEATS):
        print(f"case plan_trace decode100k repeat {k}", flush=True)
        off, peak = binding.plan_trace(*args, t.num_ops)
        assert int(peak.item()) == exp["peak"], f"repeat {k}: peak differs"
        assert _sha(host(off)) == exp["offsets_sha256"], f"repeat {k}: offsets differ"


def test_plan_trace_repeats_best_fit():
    binding = need_gpu()
    rng = np.random.default_rng(77)
    t = tg.random_trace(rng, 20000, 3000, max_len=400, sorted_first=True)
    args = (dev(t.size, torch.int64), dev(t.first, torch.int32), dev(t.last, torch.int32))
    ref = None
    for k in range(REPEATS):
        print(f"case plan_trace best fit 20000 tensors repeat {k}", flush=True)
        off, _ = binding.plan_trace(*args, t.num_ops, policy=binding.BEST_FIT)
        o = host(off)
        ref = o if ref is None else ref
        assert np.array_equal(o, ref), f"repeat {k}: offsets differ"


def test_validate_repeats_decode100k():
    binding = need_gpu()
    t, args, off = _decode_plan(binding)
    exp = _expected("decode100k_validation")
    bad, _ = tg.corrupt_offsets(t.first, t.last, off, seed=5, k=100)
    assert _sha(bad) == exp["corrupted_offsets_sha256"]
    bad_d = dev(bad, torch.int64)
    for k in range(REPEATS):
        print(f"case validate decode100k corrupted repeat {k}", flush=True)
        pairs, cnt, st = binding.validate_plan(*args, bad_d, capacity=exp["corrupted_conflicts"])
        assert cnt == exp["corrupted_conflicts"] and st == binding.MP_OK, f"repeat {k}"
        assert _sha(host(pairs)) == exp["pairs_sha256"], f"repeat {k}: pairs differ"


def test_validate_batch_repeats():
    binding = need_gpu()
    batch = tg.resnext_batch(64, 2000)
    begin, num_ops, size, first, last = batch_to_device(batch)
    off, _, _ = binding.plan_batch(begin, num_ops, size, first, last, max_trace_len=2000)
    o = host(off)
    o[5] = o[6]  # tensors 5 and 6 of trace 0 intersect: a conflict to report
    bad = dev(o, torch.int64)
    ref = None
    for k in range(REPEATS):
        for sorted_hint, max_len in ((True, 2000), (False, 0)):
            print(f"case validate_batch repeat {k} sorted={sorted_hint}", flush=True)
            pairs, cnt, st = binding.validate_batch(begin, size, first, last, bad, capacity=4096,
                                                    assume_sorted=sorted_hint,
                                                    max_trace_len=max_len)
            got = (cnt, _sha(host(pairs)))
            ref = got if ref is None else ref
            assert got == ref and cnt > 0, f"repeat {k}: differs"


def _probe_once(binding, args, off_d, num_ops, top, capacity):
    slab = torch.empty(top, dtype=torch.uint8, device="cuda")
    ws = torch.empty(binding.workspace_size(binding.OP_PROBE, int(off_d.numel()), num_ops, capacity),
                     dtype=torch.uint8, device="cuda")
    clob, cnt = binding.probe_plan(*args, off_d, num_ops, slab, workspace=ws)
    return host(clob), int(cnt.item()), int(host(ws[:12].view(torch.int32))[2])


def test_probe_repeats_tiled_decode100k():
    binding = need_gpu()
    t, args, off = _decode_plan(binding)
    bad, _ = tg.corrupt_offsets(t.first, t.last, off, seed=5, k=100)
    top = int((bad + t.size).max())
    ref = None
    for k in range(REPEATS):
        print(f"case probe tiled decode100k corrupted repeat {k}", flush=True)
        clob, cnt, ran_ops = _probe_once(binding, args, dev(bad, torch.int64), t.num_ops, top, 0)
        assert ran_ops == 0 and cnt > 0
        ref = (clob, cnt) if ref is None else ref
        assert cnt == ref[1] and np.array_equal(clob, ref[0]), f"repeat {k}: differs"


def test_probe_repeats_op_by_op():
    binding = need_gpu()
    rng = np.random.default_rng(78)
    t = tg.random_trace(rng, 3000, 800, max_len=40, sorted_first=True)
    args = (dev(t.size, torch.int64), dev(t.first, torch.int32), dev(t.last, torch.int32))
    off, _ = binding.plan_trace(*args, t.num_ops)
    o = host(off)
    o[::50] = 0  # some tensors moved onto others
    top = int((o + t.size).max())
    ref = None
    for k in range(REPEATS):
        print(f"case probe op by op repeat {k}", flush=True)
        clob, cnt, ran_ops = _probe_once(binding, args, dev(o, torch.int64), t.num_ops, top, 1)
        assert ran_ops == 1 and cnt > 0
        ref = (clob, cnt) if ref is None else ref
        assert cnt == ref[1] and np.array_equal(clob, ref[0]), f"repeat {k}: differs"


def test_live_profile_repeats():
    binding = need_gpu()
    t = tg.ranking1m()
    args = (dev(t.size, torch.int64), dev(t.first, torch.int32), dev(t.last, torch.int32))
    ref = None
    for k in range(REPEATS):
        print(f"case live profile ranking1m repeat {k}", flush=True)
        live, mx = binding.live_bytes_profile(*args, t.num_ops)
        got = (_sha(host(live)), int(mx.item()))
        ref = got if ref is None else ref
        assert got == ref, f"repeat {k}: differs"
