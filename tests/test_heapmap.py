"""Heap-map export (host only): rectangles match the plan, and for a valid
plan two rectangles meet only when their tensors do not conflict."""
import re

import numpy as np

import oracle
from paper_2203_00448_amd import heapmap, tracegen as tg


def test_rectangles_csv_svg():
    t = tg.chain256()
    off, peak = oracle.plan_trace(t.size, t.first, t.last, t.num_ops)
    r = heapmap.rectangles(t.size, t.first, t.last, off)
    assert r.shape == (256, 4)
    assert np.array_equal(r[:, 0], t.first) and np.array_equal(r[:, 1], t.last + 1)
    assert np.array_equal(r[:, 2], off) and int(r[:, 3].max()) == peak
    csv = heapmap.to_csv(t.size, t.first, t.last, off)
    assert csv.count("\n") == 257
    svg = heapmap.to_svg(t.size, t.first, t.last, off, title="chain256")
    assert len(re.findall(r'class="tensor"', svg)) == 256
    assert f"peak {peak} bytes" in svg


def test_rectangles_overlap_iff_conflict():
    rng = np.random.default_rng(99)
    for valid in (True, False):
        n = 40
        size = 64 * rng.integers(1, 9, n)
        first = rng.integers(0, 20, n)
        last = first + rng.integers(0, 5, n)
        T = int(last.max()) + 1
        off = oracle.plan_trace(size, first, last, T)[0] if valid else \
            64 * rng.integers(0, 30, n)
        r = heapmap.rectangles(size, first, last, off)
        meet = [(i, j) for i in range(n) for j in range(i + 1, n)
                if r[i, 0] < r[j, 1] and r[j, 0] < r[i, 1] and r[i, 2] < r[j, 3] and r[j, 2] < r[i, 3]]
        pairs, cnt = oracle.validate_plan(size, first, last, off)
        assert sorted(meet) == sorted(map(tuple, pairs.reshape(-1, 2).tolist()))
        assert (cnt == 0) == valid
