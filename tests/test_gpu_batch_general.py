"""mp_plan_batch on traces the LDS-resident path cannot hold: the same
workgroup plans them on the general path (64-bit offsets, the greedy taken
one tensor at a time in rank order).  No valid trace is refused (Section 2.3's
problem has no bound on sizes or on how many lifetimes intersect; Eq. 2.1
only forbids overlap).  Offsets, peaks and lower bounds must match the CPU
oracle bit for bit under both fit policies."""
import numpy as np
import pytest

import oracle
from gpu_util import batch_to_device, host, need_gpu
from paper_2203_00448_amd import tracegen as tg

pytestmark = pytest.mark.gpu
POLICIES = [("lowest", oracle.LOWEST_FIT), ("best", oracle.BEST_FIT)]


def _check(binding, batch, policy, **kw):
    args = batch_to_device(batch)
    off, peak, lb = binding.plan_batch(*args, policy=policy, **kw)
    off, peak, lb = host(off), host(peak), host(lb)
    eo, ep = oracle.plan_batch(batch.begin, batch.num_ops, batch.size, batch.first, batch.last,
                               policy)
    el = np.array([oracle.live_bytes_profile(batch.trace(b).size, batch.trace(b).first,
                                             batch.trace(b).last, batch.trace(b).num_ops)[1]
                   for b in range(batch.n_traces)], dtype=np.int64)
    bad = np.nonzero(off != eo)[0]
    assert bad.size == 0, f"{bad.size} offsets differ, first at {bad[:5]}"
    assert np.array_equal(peak, ep)
    assert np.array_equal(lb, el)
    return off, peak


def _wide_pair():
    # 2^32 + 2 bytes in units of one byte: past the 31-bit unit counts of the LDS path
    return tg.Trace(np.array([2 ** 31 + 1, 2 ** 31 + 1], np.int64), np.zeros(2, np.int32),
                    np.zeros(2, np.int32), 1)


@pytest.mark.parametrize("name,policy", POLICIES)
def test_wide_sizes(name, policy):
    binding = need_gpu()
    print(f"case two tensors of 2^31 + 1 bytes and random odd 2^28..2^34-byte traces, {name}",
          flush=True)
    rng = np.random.default_rng(300)
    traces = [_wide_pair(), tg.chain256()]
    for k in range(40):
        n = int(rng.choice([1, 2, 5, 40, 300, 1000]))
        T = int(rng.integers(1, max(2, n)))
        t = tg.random_trace(rng, n, T, max_len=int(rng.integers(1, 12)), sorted_first=(k % 2 == 0))
        t.size[:] = rng.integers(2 ** 28, 2 ** 34, n) | 1   # odd: a unit of one byte
        if k % 5 == 0:
            t.size[:] = (2 ** 33 + 1) * rng.integers(1, 4, n)   # many equal sizes
        traces.append(t)
    _, peak = _check(binding, tg.concat(traces), policy, max_trace_len=1000)
    assert peak[0] == 2 * (2 ** 31 + 1)


@pytest.mark.parametrize("name,policy", POLICIES)
def test_fully_overlapping_2000(name, policy):
    """2000 tensors alive at the same op: 1,999,000 intersecting pairs, far
    past the LDS lists; offsets are the exclusive prefix sums in rank order."""
    binding = need_gpu()
    print(f"case 2000 fully overlapping tensors, {name}", flush=True)
    rng = np.random.default_rng(301)
    n = 2000
    full = tg.Trace(64 * rng.integers(1, 5000, n), np.zeros(n, np.int32), np.zeros(n, np.int32), 1)
    off, peak = _check(binding, tg.concat([full, tg.resnext_trace(3)]), policy,
                       max_trace_len=2000)
    assert peak[0] == int(full.size.sum())


@pytest.mark.parametrize("name,policy", POLICIES)
def test_star_300(name, policy):
    """One tensor alive through every op meets the 299 others (each alive at
    one op): more than the 256 neighbours BEST_FIT fits in one wave."""
    binding = need_gpu()
    print(f"case star of 300, {name}", flush=True)
    n = 300
    t = tg.Trace(np.full(n, 64, np.int64), np.arange(n, dtype=np.int32),
                 np.arange(n, dtype=np.int32), n)
    t.first[0], t.last[0] = 0, n - 1
    _, peak = _check(binding, tg.concat([t]), policy)
    assert peak[0] == 128


@pytest.mark.parametrize("name,policy", POLICIES)
def test_long_tensors(name, policy):
    """Tensors that meet others born more than 223 positions later are named
    through a table of 32 slots: 1, 32 and 33 such tensors (the last takes
    the general path), long-lived ones among chains of short ones."""
    binding = need_gpu()
    print(f"case long-lived tensors in 1200-tensor traces, {name}", flush=True)
    rng = np.random.default_rng(302)
    traces = []
    for n_long in (1, 31, 32, 33, 60):
        n = 1200
        first = np.arange(n, dtype=np.int32)
        last = np.minimum(n - 1, first + rng.integers(0, 4, n)).astype(np.int32)
        picks = rng.choice(n - 300, n_long, replace=False)
        last[picks] = np.minimum(n - 1, picks + rng.integers(230, 900, n_long))
        size = 64 * rng.integers(1, 200, n)
        traces.append(tg.Trace(size, first, last, n))
    _check(binding, tg.concat(traces), policy, max_trace_len=1200)


@pytest.mark.parametrize("name,policy", POLICIES)
def test_pair_capacity_boundary(name, policy):
    """Traces with exactly the LDS list capacity of intersecting pairs and one
    more (that one takes the general path)."""
    binding = need_gpu()
    cap = binding.batch_pair_capacity(64)
    print(f"case pair capacity {cap} and {cap + 1} at max_trace_len 64, {name}", flush=True)
    assert cap >= 64 * 63 // 2    # every pair of a 64-tensor trace fits
    cap = binding.batch_pair_capacity(2000)
    rng = np.random.default_rng(303)
    traces = []
    for extra in (0, 1):
        # one birth per op, band lengths (tensors met later) summing to cap + extra
        n = 2000
        room = n - 1 - np.arange(n)
        band = np.minimum(np.full(n, cap // n, np.int64), room)
        short = cap + extra - int(band.sum())
        grow = np.nonzero(band < room)[0][:short]
        band[grow] += 1
        first = np.arange(n, dtype=np.int32)
        last = (first + band).astype(np.int32)
        last = np.minimum(last, n - 1).astype(np.int32)
        t = tg.Trace(64 * rng.integers(1, 100, n), first, last, n)
        pairs = int((np.searchsorted(first, last, side="right") - np.arange(n) - 1).sum())
        traces.append((pairs, t))
    assert traces[1][0] == traces[0][0] + 1 and traces[0][0] <= cap < traces[1][0]
    _check(binding, tg.concat([t for _, t in traces]), policy, max_trace_len=2000)
