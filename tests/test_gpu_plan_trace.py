"""Parity of the single-trace HIP planner (mp_plan_trace) with the CPU oracle.

Offsets and the peak must match bit for bit.  The two largest traces use
reference digests written by tests/golden/make_expected.py (oracle only)."""
import hashlib
import json
import os

import numpy as np
import pytest

import oracle
from defs import interleaved_trace, packed_wide_trace
from gpu_util import dev, host, need_gpu, torch
from paper_2203_00448_amd import tracegen as tg

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def _expected(name):
    with open(os.path.join(HERE, "golden", "expected.json")) as fh:
        return json.load(fh)["configs"][name]


def _sha(a):
    return hashlib.sha256(np.ascontiguousarray(a).astype("<i8").tobytes()).hexdigest()


def _plan(binding, t, **kw):
    off, peak = binding.plan_trace(dev(t.size, torch.int64), dev(t.first, torch.int32),
                                   dev(t.last, torch.int32), t.num_ops, **kw)
    return host(off), int(peak.item())


def _check(binding, t):
    off, peak = _plan(binding, t)
    eo, ep = oracle.plan_trace(t.size, t.first, t.last, t.num_ops)
    bad = np.nonzero(off != eo)[0]
    assert bad.size == 0, f"{bad.size} offsets differ, first at {bad[:5]}"
    assert peak == ep


def test_chain256():
    binding = need_gpu()
    print("case chain256", flush=True)
    _check(binding, tg.chain256())


def test_random_traces():
    binding = need_gpu()
    rng = np.random.default_rng(300)
    print("case random traces", flush=True)
    for k in range(24):
        n = int(rng.choice([1, 2, 3, 40, 700, 5000]))
        T = int(rng.integers(1, 2000))
        alphabet = [64, 128, 192, 448, 4096] if k % 3 == 0 else None
        t = tg.random_trace(rng, n, T, max_len=int(rng.integers(1, T + 1)), sizes=alphabet,
                            sorted_first=(k % 2 == 0))
        _check(binding, t)
    # ranks are handed out in blocks of 32 per XCD, one rank per workgroup:
    # traces ending at and around a block, two blocks and the grid
    print("case rank-block boundaries", flush=True)
    for n in [31, 32, 33, 63, 64, 65, 255, 256, 257, 1025]:
        t = tg.random_trace(rng, n, max(2, n // 3), max_len=8, sizes=[64, 192, 448])
        _check(binding, t)


def test_sort_path_boundaries():
    """Sorts of up to 4,096 pairs take one workgroup's sort in LDS, longer ones
    digit passes: unsorted traces on both sides of that size, with few sizes
    (ties keep position order) and with one-byte units (odd sizes of
    2^28..2^34 bytes, so the rank keys are 64 bits wide)."""
    binding = need_gpu()
    rng = np.random.default_rng(302)
    for n in [4095, 4096, 4097]:
        print(f"case unsorted, {n} tensors, three sizes", flush=True)
        _check(binding, tg.random_trace(rng, n, n // 4, max_len=30, sizes=[64, 192, 448]))
        print(f"case unsorted, {n} tensors, 64-bit unit counts", flush=True)
        t = tg.random_trace(rng, n, n // 4, max_len=30)
        t.size[:] = rng.integers(2 ** 28, 2 ** 34, n) | 1
        t.size[::3] = 2 ** 33 + 1
        _check(binding, t)


def test_adversarial_shapes():
    binding = need_gpu()
    rng = np.random.default_rng(301)
    print("case full overlap, 9000 tensors", flush=True)
    # up to 8999 placed predecessors, drawn as one coverage bitmap; every
    # lower rank is a predecessor, so a tensor can find ~500 of them unplaced
    # (held by other workgroups, or untaken in other XCDs' rank blocks), the
    # most the wait holds (a broken bound raises the device status)
    n = 9000
    _check(binding, tg.Trace(64 * rng.integers(1, 200, n), np.zeros(n, np.int32),
                             np.full(n, 3, np.int32), 4))
    print("case equal sizes / long-lived / disjoint", flush=True)
    _check(binding, tg.random_trace(rng, 6000, 3000, max_len=20, sizes=[320]))
    t = tg.random_trace(rng, 8000, 4000, max_len=4, sorted_first=True)
    t.last[::50] = 3999  # 160 long-lived tensors
    _check(binding, t)
    n = 3000
    _check(binding, tg.Trace(64 * rng.integers(1, 50, n), np.arange(n, dtype=np.int32),
                             np.arange(n, dtype=np.int32), n))


def test_union_fallbacks():
    """Predecessor sets the coverage bitmap declines take the sorted runs:
    more than 16,384 disjoint intervals, and a union wider than 2^20 units
    (with more than 16,384 ranges, so two runs)."""
    binding = need_gpu()
    for name, (sz, f, l, T, eo, ep) in [("more intervals than one run", interleaved_trace(16400)),
                                        ("union wider than the bitmap", packed_wide_trace(16600))]:
        print("case", name, flush=True)
        off, peak = _plan(binding, tg.Trace(sz, f, l, T))
        bad = np.nonzero(off != eo)[0]
        assert bad.size == 0, f"{name}: {bad.size} offsets differ, first at {bad[:5]}"
        assert peak == ep


def test_decode100k():
    binding = need_gpu()
    t = tg.decode100k()
    exp = _expected("decode100k")
    print("case decode100k", flush=True)
    off, peak = _plan(binding, t)
    assert peak == exp["peak"]
    assert _sha(off) == exp["offsets_sha256"]
    off2, _ = _plan(binding, t)
    assert np.array_equal(off, off2)  # repeatable


def test_ranking1m():
    binding = need_gpu()
    t = tg.ranking1m()
    exp = _expected("ranking1m")
    print("case ranking1m", flush=True)
    off, peak = _plan(binding, t)
    assert peak == exp["peak"]
    assert _sha(off) == exp["offsets_sha256"]


def test_debug_wait_paths(monkeypatch):
    """The test build of the library (MP_DEBUG_WAIT) with MEMOPLAN_DEBUG_WAIT
    drives the late-predecessor paths the schedule rarely reaches: "wide"
    holds eight late predecessors a lane in every wait, "tight" caps the late
    list at 8 so that tensors with more wait for the rest during their
    collection (reporting MP_EDEVICE).  Offsets stay exact either way."""
    binding = need_gpu()
    saved = binding._lib
    binding._lib = None
    binding.load_library(binding.DBG_WAIT_LIB_PATH)
    try:
        _debug_wait_cases(binding, monkeypatch)
    finally:
        binding._lib = saved


def _debug_wait_cases(binding, monkeypatch):
    t = tg.decode100k()
    exp = _expected("decode100k")
    monkeypatch.setenv("MEMOPLAN_DEBUG_WAIT", "wide")
    print("case decode100k, widest wait", flush=True)
    off, peak = _plan(binding, t)
    assert peak == exp["peak"] and _sha(off) == exp["offsets_sha256"]
    rng = np.random.default_rng(303)
    n = 3000
    full = tg.Trace(64 * rng.integers(1, 200, n), np.zeros(n, np.int32), np.full(n, 3, np.int32), 4)
    print("case full overlap, widest wait", flush=True)
    _check(binding, full)
    monkeypatch.setenv("MEMOPLAN_DEBUG_WAIT", "tight")
    for name, tr in [("full overlap", full),
                     ("random", tg.random_trace(rng, 5000, 600, max_len=40, sorted_first=True))]:
        print(f"case {name}, late list of 8", flush=True)
        st = binding.new_status()
        off, peak = _plan(binding, tr, check=False, status=st)
        eo, ep = oracle.plan_trace(tr.size, tr.first, tr.last, tr.num_ops)
        assert np.array_equal(off, eo) and peak == ep
        assert int(st.item()) == binding.MP_EDEVICE


def test_status_codes_and_empty():
    binding = need_gpu()
    off, peak = _plan(binding, tg.Trace(np.zeros(0, np.int64), np.zeros(0, np.int32),
                                        np.zeros(0, np.int32), 0))
    assert off.shape == (0,) and peak == 0

    def status(t):
        st = binding.new_status()
        binding.plan_trace(dev(t.size, torch.int64), dev(t.first, torch.int32),
                           dev(t.last, torch.int32), t.num_ops, check=False, status=st)
        return int(st.item())

    good = tg.chain256()
    assert status(good) == binding.MP_OK
    bad = tg.Trace(good.size.copy(), good.first.copy(), good.last.copy(), good.num_ops)
    bad.size[9] = -5
    assert status(bad) == binding.MP_EINVAL
    big = tg.Trace(np.array([2 ** 62, 2 ** 62], np.int64), np.zeros(2, np.int32),
                   np.zeros(2, np.int32), 1)
    assert status(big) == binding.MP_EOVERFLOW
    # sizes past 32-bit unit counts are planned (64-bit path), not refused
    wide = tg.Trace(np.array([2 ** 31 + 1, 2 ** 31 + 1], np.int64), np.zeros(2, np.int32),
                    np.zeros(2, np.int32), 1)
    assert status(wide) == binding.MP_OK
