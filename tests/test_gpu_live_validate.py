"""Parity of the liveness profile and plan validation kernels with the oracle."""
import json
import os

import numpy as np
import pytest

import oracle
from gpu_util import dev, host, need_gpu, torch
from paper_2203_00448_amd import tracegen as tg

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def _expected():
    path = os.path.join(HERE, "golden", "expected.json")
    with open(path) as fh:
        return json.load(fh)["configs"]


def _trace_dev(t):
    return dev(t.size, torch.int64), dev(t.first, torch.int32), dev(t.last, torch.int32)


def _sha(a):
    import hashlib
    return hashlib.sha256(np.ascontiguousarray(a).astype("<i8").tobytes()).hexdigest()


# ------------------------------------------------------------------ liveness

def test_live_profile_random():
    binding = need_gpu()
    rng = np.random.default_rng(200)
    print("case random live profiles", flush=True)
    for k in range(40):
        T = int(rng.choice([1, 2, 7, 64, 1000, 5000]))
        n = int(rng.choice([0, 1, 5, 300, 3000]))
        t = tg.random_trace(rng, n, T, max_len=int(rng.integers(1, T + 1)))
        live, mx = binding.live_bytes_profile(*_trace_dev(t), T)
        ref, rmx = oracle.live_bytes_profile(t.size, t.first, t.last, T)
        assert np.array_equal(host(live), ref), k
        assert int(mx.item()) == rmx


def test_live_profile_empty():
    binding = need_gpu()
    e = np.zeros(0, np.int64)
    live, mx = binding.live_bytes_profile(dev(e, torch.int64), dev(e, torch.int32),
                                          dev(e, torch.int32), 0)
    assert live.numel() == 0 and int(mx.item()) == 0


@pytest.mark.parametrize("name", ["decode100k", "ranking1m"])
def test_live_profile_full_workloads(name):
    binding = need_gpu()
    t = tg.decode100k() if name == "decode100k" else tg.ranking1m()
    print(f"case live profile {name}", flush=True)
    live, mx = binding.live_bytes_profile(*_trace_dev(t), t.num_ops)
    exp = _expected()[name]
    assert _sha(host(live)) == exp["live_sha256"]
    assert int(mx.item()) == exp["lb"]


def test_live_profile_status():
    binding = need_gpu()
    t = tg.chain256()
    bad = tg.Trace(t.size.copy(), t.first.copy(), t.last.copy(), 100)  # last >= num_ops
    st = binding.new_status()
    binding.live_bytes_profile(*_trace_dev(bad), 100, check=False, status=st)
    assert int(st.item()) == binding.MP_EINVAL
    big = tg.Trace(np.array([2 ** 62, 2 ** 62], np.int64), np.zeros(2, np.int32),
                   np.zeros(2, np.int32), 1)
    st = binding.new_status()
    binding.live_bytes_profile(*_trace_dev(big), 1, check=False, status=st)
    assert int(st.item()) == binding.MP_EOVERFLOW


# ------------------------------------------------------------------ validation

def _oracle_pairs(t, off, capacity=None):
    pairs, cnt = oracle.validate_plan(t.size, t.first, t.last, off, capacity)
    return pairs, cnt


def _gpu_pairs(binding, t, off, capacity=None):
    pairs, cnt, st = binding.validate_plan(*_trace_dev(t), dev(off, torch.int64),
                                           capacity=capacity)
    return host(pairs), cnt, st


def test_validate_random_sorted_and_unsorted():
    binding = need_gpu()
    rng = np.random.default_rng(201)
    print("case random validation", flush=True)
    for k in range(30):
        n = int(rng.choice([1, 2, 50, 400, 2500]))
        T = int(rng.integers(1, 200))
        t = tg.random_trace(rng, n, T, max_len=int(rng.integers(1, 60)), sorted_first=(k % 2 == 0))
        off = 64 * rng.integers(0, 40, n)  # many accidental overlaps
        ep, ec = _oracle_pairs(t, off)
        gp, gc, st = _gpu_pairs(binding, t, off, capacity=max(ec, 1))
        assert st == binding.MP_OK and gc == ec, k
        assert np.array_equal(gp, ep), k


def test_validate_sort_path_boundaries():
    """Unsorted plans on both sides of the 4,096-element single-workgroup sort:
    the position sort (n tensors) and the pair sort (capacity entries)."""
    binding = need_gpu()
    rng = np.random.default_rng(203)
    for n in [4095, 4096, 4097]:
        t = tg.random_trace(rng, n, n // 8, max_len=4)
        for spread in (3000, 500):
            off = 64 * rng.integers(0, spread, n)
            ep, ec = _oracle_pairs(t, off)
            print(f"case unsorted validation, {n} tensors ({ec} conflicts)", flush=True)
            for cap in sorted({min(ec, 4096), ec, 4097}):
                gp, gc, st = _gpu_pairs(binding, t, off, capacity=cap)
                want = binding.MP_OK if cap >= ec else binding.MP_ENOSPC
                assert st == want and gc == ec and np.array_equal(gp, ep[:cap]), (n, cap)


def test_validate_long_rows_and_capacity():
    binding = need_gpu()
    rng = np.random.default_rng(202)
    n = 3000
    t = tg.random_trace(rng, n, 600, max_len=3, sorted_first=True)
    t.first[::97] = 0                      # long-lived tensors: rows far longer than 64
    t.last[::97] = 599
    order = np.lexsort((np.arange(n), t.first))
    t = tg.Trace(t.size[order], t.first[order], t.last[order], t.num_ops)
    off = 64 * rng.integers(0, 30, n)
    ep, ec = _oracle_pairs(t, off)
    print(f"case long rows ({ec} conflicts)", flush=True)
    gp, gc, st = _gpu_pairs(binding, t, off, capacity=ec)
    assert st == binding.MP_OK and gc == ec and np.array_equal(gp, ep)
    cap = ec // 3
    gp, gc, st = _gpu_pairs(binding, t, off, capacity=cap)
    assert st == binding.MP_ENOSPC and gc == ec and np.array_equal(gp, ep[:cap])
    gp, gc, st = _gpu_pairs(binding, t, off, capacity=0)
    assert gc == ec and gp.shape[0] == 0


def test_validate_long_rows_wide_offsets():
    """Long rows whose byte ranges straddle 2^32 and lie far above it: the
    count pass compares 64-bit ranges (the 32-bit compares are used only when
    every offset + size is below 2^32); sorted and unsorted positions."""
    binding = need_gpu()
    rng = np.random.default_rng(207)
    n = 3000
    t = tg.random_trace(rng, n, 600, max_len=3, sorted_first=True)
    t.first[::89] = 0
    t.last[::89] = 599
    order = np.lexsort((np.arange(n), t.first))
    t = tg.Trace(t.size[order], t.first[order], t.last[order], t.num_ops)
    for base in ((1 << 32) - 1000, 1 << 40):
        off = base + 64 * rng.integers(0, 30, n)
        ep, ec = _oracle_pairs(t, off)
        print(f"case wide offsets base {base} ({ec} conflicts)", flush=True)
        gp, gc, st = _gpu_pairs(binding, t, off, capacity=max(ec, 1))
        assert st == binding.MP_OK and gc == ec and np.array_equal(gp, ep)
        perm = rng.permutation(n)
        tp = tg.Trace(t.size[perm], t.first[perm], t.last[perm], t.num_ops)
        ep2, ec2 = _oracle_pairs(tp, off[perm])
        gp2, gc2, st2 = _gpu_pairs(binding, tp, off[perm], capacity=max(ec2, 1))
        assert st2 == binding.MP_OK and gc2 == ec2 == ec and np.array_equal(gp2, ep2)


def test_validate_oracle_plans_are_clean():
    binding = need_gpu()
    rng = np.random.default_rng(203)
    for k in range(10):
        t = tg.random_trace(rng, 1500, 300, max_len=20, sorted_first=(k % 2 == 1))
        off, _ = oracle.plan_trace(t.size, t.first, t.last, t.num_ops)
        _, gc, st = _gpu_pairs(binding, t, off, capacity=16)
        assert gc == 0 and st == binding.MP_OK


def test_validate_decode100k_clean_and_corrupted():
    binding = need_gpu()
    t = tg.decode100k()
    exp = _expected()["decode100k_validation"]
    off, _ = oracle.plan_trace(t.size, t.first, t.last, t.num_ops)  # a few seconds on one core
    print("case decode100k validation", flush=True)
    _, gc, st = _gpu_pairs(binding, t, off, capacity=1024)
    assert gc == 0 and st == binding.MP_OK
    bad, chosen = tg.corrupt_offsets(t.first, t.last, off, seed=5, k=100)
    assert _sha(bad) == exp["corrupted_offsets_sha256"]
    gp, gc, st = _gpu_pairs(binding, t, bad, capacity=exp["corrupted_conflicts"])
    assert gc == exp["corrupted_conflicts"] and st == binding.MP_OK
    assert _sha(gp) == exp["pairs_sha256"]
    assert set(chosen.tolist()) <= set(gp.ravel().tolist())


def test_validate_batch_matches_per_trace():
    binding = need_gpu()
    rng = np.random.default_rng(204)
    traces = [tg.random_trace(rng, int(rng.choice([0, 1, 30, 700])), 100, max_len=8,
                              sorted_first=(k % 3 != 0)) for k in range(25)]
    batch = tg.concat(traces)
    off = 64 * rng.integers(0, 20, batch.size.shape[0])
    expect = []
    for b, t in enumerate(traces):
        lo = int(batch.begin[b])
        p, _ = oracle.validate_plan(t.size, t.first, t.last, off[lo:lo + t.n])
        expect.append(p + lo)
    expect = np.concatenate(expect) if expect else np.zeros((0, 2), np.int64)
    print(f"case batch validation ({expect.shape[0]} conflicts)", flush=True)
    pairs, cnt, st = binding.validate_batch(dev(batch.begin, torch.int64),
                                            dev(batch.size, torch.int64),
                                            dev(batch.first, torch.int32),
                                            dev(batch.last, torch.int32), dev(off, torch.int64),
                                            capacity=max(1, expect.shape[0]))
    assert st == binding.MP_OK and cnt == expect.shape[0]
    assert np.array_equal(host(pairs), expect)
    # past the capacity: the lexicographically first pairs (some traces are
    # unsorted, so position order differs from id order)
    for cap in (expect.shape[0] // 3, 1):
        pairs, cnt, st = binding.validate_batch(dev(batch.begin, torch.int64),
                                                dev(batch.size, torch.int64),
                                                dev(batch.first, torch.int32),
                                                dev(batch.last, torch.int32),
                                                dev(off, torch.int64), capacity=cap)
        assert st == binding.MP_ENOSPC and cnt == expect.shape[0], cap
        assert np.array_equal(host(pairs), expect[:cap]), cap


def test_validate_batch_long_rows_across_traces():
    """Batches whose traces hold long-lived tensors (bands far over 64
    candidates): the long rows of different traces share chunks of the count
    pass, and each row stays inside its own trace."""
    binding = need_gpu()
    rng = np.random.default_rng(208)
    traces = []
    for k in range(12):
        n = int(rng.choice([1, 200, 900, 1500]))
        t = tg.random_trace(rng, n, 300, max_len=4, sorted_first=(k % 4 != 0))
        t.first[::53] = 0
        t.last[::53] = 299
        traces.append(t)
    batch = tg.concat(traces)
    off = 64 * rng.integers(0, 25, batch.size.shape[0])
    expect = _batch_expect(traces, batch, off)
    print(f"case batch long rows ({expect.shape[0]} conflicts)", flush=True)
    pairs, cnt, st = binding.validate_batch(*_batch_dev(batch, off), capacity=max(1, expect.shape[0]))
    assert st == binding.MP_OK and cnt == expect.shape[0]
    assert np.array_equal(host(pairs), expect)


def _batch_expect(traces, batch, off):
    expect = []
    for b, t in enumerate(traces):
        lo = int(batch.begin[b])
        p, _ = oracle.validate_plan(t.size, t.first, t.last, off[lo:lo + t.n])
        expect.append(p + lo)
    return np.concatenate(expect) if expect else np.zeros((0, 2), np.int64)


def _batch_dev(batch, off):
    return (dev(batch.begin, torch.int64), dev(batch.size, torch.int64),
            dev(batch.first, torch.int32), dev(batch.last, torch.int32), dev(off, torch.int64))


@pytest.mark.parametrize("max_len", [700, 2048, 4096])
def test_validate_batch_per_trace_path(max_len):
    """Sorted traces with a length bound: one workgroup per trace."""
    binding = need_gpu()
    rng = np.random.default_rng(206 + max_len)
    sizes = [0, 1, 2, 31, 511, 512, 513, 700]
    traces = [tg.random_trace(rng, int(rng.choice(sizes)), 300, max_len=int(rng.integers(1, 40)),
                              sorted_first=True) for _ in range(60)]
    traces.append(tg.random_trace(rng, 700, 50, max_len=50, sorted_first=True))  # dense rows
    batch = tg.concat(traces)
    off = 64 * rng.integers(0, 30, batch.size.shape[0])
    expect = _batch_expect(traces, batch, off)
    print(f"case per-trace batch validation max_len={max_len} ({expect.shape[0]} conflicts)",
          flush=True)
    pairs, cnt, st = binding.validate_batch(*_batch_dev(batch, off), capacity=expect.shape[0],
                                            assume_sorted=True, max_trace_len=max_len)
    assert st == binding.MP_OK and cnt == expect.shape[0]
    assert np.array_equal(host(pairs), expect)
    # a smaller capacity keeps the first pairs in order and reports ENOSPC
    k = expect.shape[0] // 3
    pairs, cnt, st = binding.validate_batch(*_batch_dev(batch, off), capacity=max(k, 1),
                                            assume_sorted=True, max_trace_len=max_len)
    assert st == binding.MP_ENOSPC and cnt == expect.shape[0]
    assert np.array_equal(host(pairs), expect[:max(k, 1)])


def test_validate_batch_per_trace_sparse_ops():
    """Traces whose first ops span more than three times the trace bound
    find their bands by galloping search, the others from a table over the
    ops; one batch mixes both."""
    binding = need_gpu()
    rng = np.random.default_rng(212)
    traces = []
    for k in range(24):
        n = int(rng.integers(1, 600))
        T = int(rng.choice([4, 300, 5000, 40000]))  # 5000 and 40000: wider than 3 x 600 slots
        traces.append(tg.random_trace(rng, n, T, max_len=int(rng.integers(1, max(2, T // 8))),
                                      sorted_first=True))
    batch = tg.concat(traces)
    off = 64 * rng.integers(0, 40, batch.size.shape[0])
    expect = _batch_expect(traces, batch, off)
    print(f"case per-trace validation, sparse and dense ops ({expect.shape[0]} conflicts)",
          flush=True)
    pairs, cnt, st = binding.validate_batch(*_batch_dev(batch, off), capacity=expect.shape[0],
                                            assume_sorted=True, max_trace_len=600)
    assert st == binding.MP_OK and cnt == expect.shape[0]
    assert np.array_equal(host(pairs), expect)


def test_validate_batch_per_trace_clean_plans():
    """Oracle plans have no conflicts: the count pass alone decides."""
    binding = need_gpu()
    traces = [tg.resnext_trace(b) for b in range(6)] + [tg.chain256()]
    batch = tg.concat(traces)
    off, _ = oracle.plan_batch(batch.begin, batch.num_ops, batch.size, batch.first, batch.last)
    print("case per-trace validation of oracle plans", flush=True)
    pairs, cnt, st = binding.validate_batch(*_batch_dev(batch, off), capacity=16,
                                            assume_sorted=True, max_trace_len=2000)
    assert st == binding.MP_OK and cnt == 0
    bad, chosen = tg.corrupt_offsets(batch.first, batch.last, off, seed=5, k=40)
    expect = _batch_expect(traces, batch, bad)
    pairs, cnt, st = binding.validate_batch(*_batch_dev(batch, bad), capacity=expect.shape[0],
                                            assume_sorted=True, max_trace_len=2000)
    assert st == binding.MP_OK and cnt == expect.shape[0]
    assert np.array_equal(host(pairs), expect)


def test_validate_batch_per_trace_errors():
    binding = need_gpu()
    rng = np.random.default_rng(209)
    print("case per-trace validation errors", flush=True)
    # a trace longer than the promised bound
    long = tg.concat([tg.random_trace(rng, 300, 100, max_len=5, sorted_first=True)])
    off = np.zeros(300, np.int64)
    st = binding.new_status()
    binding.validate_batch(*_batch_dev(long, off), capacity=4, assume_sorted=True,
                           max_trace_len=200, check=False, status=st)
    assert int(st.item()) == binding.MP_EINVAL
    # a broken sorted promise
    u = tg.random_trace(rng, 400, 100, max_len=5, sorted_first=False)
    assert (np.diff(u.first) < 0).any()
    ub = tg.concat([u])
    st = binding.new_status()
    binding.validate_batch(*_batch_dev(ub, np.arange(400, dtype=np.int64) * 64), capacity=1 << 16,
                           assume_sorted=True, max_trace_len=512, check=False, status=st)
    assert int(st.item()) == binding.MP_EINVAL
    # many empty traces (more traces than tensors)
    traces = [tg.Trace(np.zeros(0, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32), 0)
              for _ in range(5000)]
    traces[17] = tg.random_trace(rng, 40, 10, max_len=5, sorted_first=True)
    batch = tg.concat(traces)
    off = 64 * rng.integers(0, 4, 40)
    expect = _batch_expect(traces, batch, off)
    pairs, cnt, st = binding.validate_batch(*_batch_dev(batch, off), capacity=max(1, expect.shape[0]),
                                            assume_sorted=True, max_trace_len=64)
    assert st == binding.MP_OK and cnt == expect.shape[0]
    assert np.array_equal(host(pairs), expect)


def test_validate_status_codes():
    binding = need_gpu()
    t = tg.chain256()
    off, _ = oracle.plan_trace(t.size, t.first, t.last, t.num_ops)
    off[3] = -64  # a negative offset is rejected (and other pairs stay within capacity)
    st = binding.new_status()
    binding.validate_plan(*_trace_dev(t), dev(off, torch.int64), capacity=8, check=False,
                          status=st)
    assert int(st.item()) == binding.MP_EINVAL


def test_validate_sorted_hint():
    binding = need_gpu()
    rng = np.random.default_rng(205)
    t = tg.random_trace(rng, 3000, 500, max_len=10, sorted_first=True)
    off = 64 * rng.integers(0, 20, t.n)
    ep, ec = _oracle_pairs(t, off)
    pairs, cnt, st = binding.validate_plan(*_trace_dev(t), dev(off, torch.int64), capacity=ec,
                                           assume_sorted=True)
    assert st == binding.MP_OK and cnt == ec and np.array_equal(host(pairs), ep)
    u = tg.random_trace(rng, 500, 100, max_len=10, sorted_first=False)
    st = binding.new_status()
    binding.validate_plan(*_trace_dev(u), dev(np.zeros(u.n, np.int64), torch.int64),
                          capacity=1 << 16, assume_sorted=True, check=False, status=st)
    assert int(st.item()) == binding.MP_EINVAL  # promise broken
