"""Parity of the other planning strategies of Section 2.3 on the GPU with
the CPU oracle: bump_allocation (offsets bit-exact) and the optimum of
Eq. 2.1 for tiny traces (the optimal peak is unique and must match exactly;
optimal plans are not, so the GPU's plan is checked to be valid and to reach
that peak)."""
import json
import os

import numpy as np
import pytest

import oracle
from gpu_util import batch_to_device, dev, host, need_gpu, torch
from paper_2203_00448_amd import tracegen as tg

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def _tiny(rng, n, T=6, span=4, unit=64, kinds=8):
    size = unit * rng.integers(1, kinds, n)
    first = rng.integers(0, T, n)
    last = first + rng.integers(0, span, n)
    return tg.Trace(size.astype(np.int64), first.astype(np.int32), last.astype(np.int32),
                    int(last.max()) + 1 if n else 1)


def _bump(binding, t, **kw):
    o, p = binding.bump_plan(dev(t.size, torch.int64), dev(t.first, torch.int32),
                             dev(t.last, torch.int32), t.num_ops, **kw)
    return host(o), host(p)


def test_bump_hand_case_and_random_traces():
    binding = need_gpu()
    print("case bump: hand case, random single traces", flush=True)
    t = tg.Trace(np.array([64, 32, 16], np.int64), np.array([0, 1, 0], np.int32),
                 np.array([1, 2, 0], np.int32), 3)
    o, p = _bump(binding, t)
    assert o.tolist() == [0, 80, 64] and p.tolist() == [112]
    rng = np.random.default_rng(95)
    for n in (0, 1, 2, 255, 256, 257, 5000, 70000):
        T = max(1, n // 4)
        t = tg.random_trace(rng, n, T, max_len=8, sorted_first=bool(n % 2)) if n else \
            tg.Trace(np.zeros(0, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32), 1)
        o, p = _bump(binding, t)
        eo, ep = oracle.bump_plan(t.size, t.first, t.last, t.num_ops)
        assert np.array_equal(o, eo) and int(p[0]) == ep


def test_bump_batches_and_decode():
    binding = need_gpu()
    print("case bump: ragged batch (with empty traces), decode100k", flush=True)
    rng = np.random.default_rng(96)
    traces = []
    for k in range(300):
        n = int(rng.choice([0, 1, 3, 17, 64, 300]))
        traces.append(tg.random_trace(rng, n, max(1, n), max_len=5) if n else
                      tg.Trace(np.zeros(0, np.int64), np.zeros(0, np.int32),
                               np.zeros(0, np.int32), 1))
    b = tg.concat(traces)
    T = int(max(t.num_ops for t in traces))
    o, p = binding.bump_plan(dev(b.size, torch.int64), dev(b.first, torch.int32),
                             dev(b.last, torch.int32), T, begin=dev(b.begin, torch.int64))
    o, p = host(o), host(p)
    for k, t in enumerate(traces):
        lo, hi = int(b.begin[k]), int(b.begin[k + 1])
        eo, ep = oracle.bump_plan(t.size, t.first, t.last, t.num_ops)
        assert np.array_equal(o[lo:hi], eo) and int(p[k]) == ep
    t = tg.decode100k()
    o, p = _bump(binding, t)
    eo, ep = oracle.bump_plan(t.size, t.first, t.last, t.num_ops)
    assert np.array_equal(o, eo) and int(p[0]) == ep


def test_bump_status_codes():
    binding = need_gpu()
    print("case bump status codes", flush=True)
    for size, first, last in (([64, 0], [0, 0], [0, 0]), ([64], [1], [0]), ([64], [0], [5])):
        st = binding.new_status()
        binding.bump_plan(dev(np.array(size), torch.int64), dev(np.array(first), torch.int32),
                          dev(np.array(last), torch.int32), 2, check=False, status=st)
        assert int(st.item()) == binding.MP_EINVAL
    st = binding.new_status()
    big = np.array([2 ** 62, 2 ** 62, 2 ** 62], np.int64)
    binding.bump_plan(dev(big, torch.int64), dev(np.zeros(3), torch.int32),
                      dev(np.zeros(3), torch.int32), 1, check=False, status=st)
    assert int(st.item()) == binding.MP_EOVERFLOW
    st = binding.new_status()  # trace bounds that do not end at n
    binding.bump_plan(dev(np.full(3, 64), torch.int64), dev(np.zeros(3), torch.int32),
                      dev(np.zeros(3), torch.int32), 1, begin=dev(np.array([0, 2]), torch.int64),
                      check=False, status=st)
    assert int(st.item()) == binding.MP_EINVAL


def _optimal(binding, traces):
    b = tg.concat(traces)
    o, p = binding.optimal_batch(*batch_to_device(b))
    return b, host(o), host(p)


def _check_optimal(b, o, p, traces, expected):
    for k, t in enumerate(traces):
        lo, hi = int(b.begin[k]), int(b.begin[k + 1])
        assert int(p[k]) == expected[k], k
        if hi > lo:
            assert int((o[lo:hi] + t.size).max()) == int(p[k])
            assert oracle.validate_plan(t.size, t.first, t.last, o[lo:hi])[1] == 0


def test_optimal_hand_examples():
    binding = need_gpu()
    print("case optimal: hand examples", flush=True)
    with open(os.path.join(HERE, "golden", "hand_examples.json")) as fh:
        ex = json.load(fh)["examples"]
    traces = [tg.Trace(np.asarray(e["size"], np.int64), np.asarray(e["first"], np.int32),
                       np.asarray(e["last"], np.int32), int(max(e["last"])) + 1) for e in ex]
    b, o, p = _optimal(binding, traces)
    _check_optimal(b, o, p, traces, [e["opt"] for e in ex])


def test_optimal_random_batches():
    binding = need_gpu()
    rng = np.random.default_rng(97)
    print("case optimal: 400 random traces of 0-9 tensors, 6 of 10", flush=True)
    traces = [_tiny(rng, int(rng.integers(0, 10))) for _ in range(400)]
    traces += [_tiny(rng, 10, T=8, span=5) for _ in range(6)]
    b, o, p = _optimal(binding, traces)
    expected = [oracle.optimal_plan(t.size, t.first, t.last, t.num_ops)[1] for t in traces]
    _check_optimal(b, o, p, traces, expected)


def test_optimal_closed_forms_up_to_12():
    binding = need_gpu()
    rng = np.random.default_rng(98)
    print("case optimal: closed forms with 11 and 12 tensors", flush=True)
    traces, expected = [], []
    for n in (11, 12):
        size = 16 * rng.integers(1, 30, n)
        traces.append(tg.Trace(size, np.zeros(n, np.int32), np.full(n, 2, np.int32), 3))
        expected.append(int(size.sum()))      # every pair meets
        ops = np.arange(n, dtype=np.int32)
        traces.append(tg.Trace(size, ops, ops, n))
        expected.append(int(size.max()))      # no pair meets
        first = rng.integers(0, 8, n).astype(np.int32)
        last = (first + rng.integers(0, 4, n)).astype(np.int32)
        T = int(last.max()) + 1
        omega = max(int(((first <= t) & (t <= last)).sum()) for t in range(T))
        traces.append(tg.Trace(np.full(n, 48, np.int64), first, last, T))
        expected.append(48 * omega)           # equal sizes: interval graphs are perfect
    b, o, p = _optimal(binding, traces)
    _check_optimal(b, o, p, traces, expected)
    # random traces of 11 and 12: between the lower bound and the greedy plan
    traces = [_tiny(rng, n, T=10, span=4) for n in (11, 12, 11, 12)]
    b, o, p = _optimal(binding, traces)
    for k, t in enumerate(traces):
        lb = oracle.live_bytes_profile(t.size, t.first, t.last, t.num_ops)[1]
        greedy = oracle.plan_trace(t.size, t.first, t.last, t.num_ops)[1]
        assert lb <= int(p[k]) <= greedy
    _check_optimal(b, o, p, traces, [int(x) for x in p])


def test_optimal_status_codes():
    binding = need_gpu()
    print("case optimal status codes", flush=True)
    st = binding.new_status()
    b = tg.concat([tg.Trace(np.full(13, 64, np.int64), np.zeros(13, np.int32),
                            np.zeros(13, np.int32), 1)])
    binding.optimal_batch(*batch_to_device(b), check=False, status=st)
    assert int(st.item()) == binding.MP_EINVAL
    st = binding.new_status()
    b = tg.concat([tg.Trace(np.array([64, 0], np.int64), np.zeros(2, np.int32),
                            np.zeros(2, np.int32), 1)])
    binding.optimal_batch(*batch_to_device(b), check=False, status=st)
    assert int(st.item()) == binding.MP_EINVAL


def test_optimal_tiny_batch_workload():
    binding = need_gpu()
    print("case optimal: first 12 traces of the tiny ResNeXt-like batch (oracle ~1 s each)",
          flush=True)
    batch = tg.tiny_batch(12, 10)
    traces = [batch.trace(k) for k in range(12)]
    b, o, p = _optimal(binding, traces)
    expected = [oracle.optimal_plan(t.size, t.first, t.last, t.num_ops)[1] for t in traces]
    _check_optimal(b, o, p, traces, expected)


# ---------------------------------------------------------------------------
# Greedy by Breadth: offsets and peaks bit-exact against the oracle

def _check_breadth(binding, traces, policy):
    b = tg.concat(traces)
    o, p = binding.plan_breadth_batch(*batch_to_device(b), policy=policy)
    o, p = host(o), host(p)
    for k, t in enumerate(traces):
        lo, hi = int(b.begin[k]), int(b.begin[k + 1])
        eo, ep = oracle.plan_breadth(t.size, t.first, t.last, t.num_ops, policy)
        bad = np.nonzero(o[lo:hi] != eo)[0]
        assert bad.size == 0, f"trace {k}: {bad.size} offsets differ, first at {bad[:5]}"
        assert int(p[k]) == ep


def test_breadth_hand_case():
    binding = need_gpu()
    print("case breadth hand case", flush=True)
    t = tg.Trace(np.array([100, 10, 50, 30], np.int64), np.array([0, 1, 2, 0], np.int32),
                 np.array([1, 2, 3, 0], np.int32), 4)
    o, p = binding.plan_breadth_batch(*batch_to_device(tg.concat([t])))
    assert host(o).tolist() == [0, 100, 0, 100] and int(p.item()) == 130


@pytest.mark.parametrize("policy", [0, 1])
def test_breadth_random_ragged(policy):
    binding = need_gpu()
    rng = np.random.default_rng(130 + policy)
    print(f"case breadth random ragged batch, policy {policy}", flush=True)
    traces = []
    for k in range(120):
        n = int(rng.choice([0, 1, 2, 3, 17, 64, 150, 511, 512, 513, 2047, 2048]))
        if n <= 150:
            T, span = int(rng.integers(1, 20)), int(rng.integers(1, 20))
        else:
            T, span = n + 1, int(rng.integers(1, 12))
        alphabet = [64, 128, 192, 448, 1024] if k % 3 == 0 else None
        traces.append(tg.random_trace(rng, n, T, max_len=span, sizes=alphabet) if n else
                      tg.Trace(np.zeros(0, np.int64), np.zeros(0, np.int32),
                               np.zeros(0, np.int32), 1))
    # dense traces: hundreds of placed neighbours per tensor (beyond one wave)
    traces += [tg.random_trace(rng, 600, 20, max_len=20), tg.random_trace(rng, 2000, 40, max_len=40)]
    _check_breadth(binding, traces, policy)


def test_breadth_resnext_and_tiny():
    binding = need_gpu()
    print("case breadth: 16 ResNeXt-like traces of 2000, 64 tiny traces", flush=True)
    _check_breadth(binding, [tg.resnext_trace(b) for b in range(16)], 0)
    tiny = tg.tiny_batch(64, 10)
    _check_breadth(binding, [tiny.trace(k) for k in range(64)], 1)


def test_breadth_status_codes():
    binding = need_gpu()
    print("case breadth status codes", flush=True)
    for t in (tg.Trace(np.full(2049, 64, np.int64), np.zeros(2049, np.int32),
                       np.zeros(2049, np.int32), 1),
              tg.Trace(np.array([64, 0], np.int64), np.zeros(2, np.int32),
                       np.zeros(2, np.int32), 1)):
        st = binding.new_status()
        binding.plan_breadth_batch(*batch_to_device(tg.concat([t])), check=False, status=st)
        assert int(st.item()) == binding.MP_EINVAL
