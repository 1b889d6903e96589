"""mp_plan_trace on traces beyond the 32-bit fast path: sizes summing to 2^32
units or more (the 64-bit placement kernel) and tensors with more than
131,072 earlier-ranked intersecting tensors (a shared pool buffer and the
general sort-and-merge fit).  Section 2.3's problem bounds neither; offsets
and peaks must match the CPU oracle bit for bit under both fit policies."""
import numpy as np
import pytest

import oracle
from gpu_util import dev, host, need_gpu, torch
from paper_2203_00448_amd import tracegen as tg

pytestmark = pytest.mark.gpu
POLICIES = [("lowest", oracle.LOWEST_FIT), ("best", oracle.BEST_FIT)]


def _check(binding, t, policy):
    off, peak = binding.plan_trace(dev(t.size, torch.int64), dev(t.first, torch.int32),
                                   dev(t.last, torch.int32), t.num_ops, policy=policy)
    off, peak = host(off), int(peak.item())
    eo, ep = oracle.plan_trace(t.size, t.first, t.last, t.num_ops, policy)
    bad = np.nonzero(off != eo)[0]
    assert bad.size == 0, f"{bad.size} offsets differ, first at {bad[:5]}"
    assert peak == ep
    return off, peak


def _odd_sizes(rng, n):
    return rng.integers(2 ** 28, 2 ** 34, n) | 1   # odd: a unit of one byte, sums past 2^32


@pytest.mark.parametrize("name,policy", POLICIES)
def test_wide_pair_and_random(name, policy):
    binding = need_gpu()
    print(f"case wide pair and random wide traces, {name}", flush=True)
    pair = tg.Trace(np.array([2 ** 31 + 1, 2 ** 31 + 1], np.int64), np.zeros(2, np.int32),
                    np.zeros(2, np.int32), 1)
    off, peak = _check(binding, pair, policy)
    assert sorted(off.tolist()) == [0, 2 ** 31 + 1] and peak == 2 ** 32 + 2
    rng = np.random.default_rng(500)
    for k in range(10):
        n = int(rng.choice([3, 50, 700, 5000]))
        T = int(rng.integers(1, 1500))
        t = tg.random_trace(rng, n, T, max_len=int(rng.integers(1, T + 1)),
                            sorted_first=(k % 2 == 0))
        t.size[:] = _odd_sizes(rng, n)
        if k % 3 == 0:
            t.size[:] = (2 ** 33 + 1) * rng.integers(1, 4, n)   # ties
        _check(binding, t, policy)


@pytest.mark.parametrize("name,policy", POLICIES)
def test_wide_full_overlap_merges(name, policy):
    """9000 fully overlapping tensors with 64-bit unit counts: the last ones
    have more predecessors than one LDS run of 8192 (sorted runs merged)."""
    binding = need_gpu()
    print(f"case 9000 fully overlapping wide tensors, {name}", flush=True)
    rng = np.random.default_rng(501)
    n = 9000
    t = tg.Trace(_odd_sizes(rng, n), np.zeros(n, np.int32), np.full(n, 2, np.int32), 3)
    off, peak = _check(binding, t, policy)
    assert peak == int(t.size.sum())


def _star(rng, m, wide):
    """m ops; at op i a large tensor B_i and a middle one L_i (alive at op i
    only), and one small tensor alive at every op: it ranks last and meets all
    2m others, far past 131,072."""
    n = 2 * m + 1
    size = np.empty(n, np.int64)
    first = np.empty(n, np.int32)
    size[0:2 * m:2] = 64 * rng.integers(200, 400, m)
    size[1:2 * m:2] = 64 * rng.integers(2, 199, m)
    first[0:2 * m:2] = np.arange(m)
    first[1:2 * m:2] = np.arange(m)
    size[-1], first[-1] = 64, 0
    last = first.copy()
    last[-1] = m - 1
    if wide:
        size += 1   # odd sizes: one-byte unit, 64-bit counts
        size[:4] += 2 ** 34
    return tg.Trace(size, first, last, m)


@pytest.mark.parametrize("wide", [False, True])
@pytest.mark.parametrize("name,policy", POLICIES)
def test_more_than_131072_predecessors(name, policy, wide):
    binding = need_gpu()
    print(f"case star of 280,001 tensors (280,000 predecessors), wide={wide}, {name}", flush=True)
    rng = np.random.default_rng(502)
    t = _star(rng, 140_000, wide)
    off, peak = _check(binding, t, policy)
    ends = t.size[:-1] + off[:-1]
    assert off[-1] == ends.max()   # the union of its predecessors is one interval from 0
