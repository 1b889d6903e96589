"""Parity of the plan-application probe on the GPU with the CPU oracle.

The plan applied as in Section 3.3 (one slab, every tensor a view at its
offset, Listing 5) and exercised by replaying the ops: each tensor writes
id + 1 into its words at its first op (the larger value kept), checks them at
its last op and clears them.  Which tensors find a foreign word is integer
work and does not depend on the order of one op's writers, so the GPU result
must equal the oracle's bit for bit.
"""
import numpy as np
import pytest

import oracle
from gpu_util import dev, host, need_gpu, torch
from paper_2203_00448_amd import tracegen as tg

pytestmark = pytest.mark.gpu


def _probe(binding, size, first, last, off, num_ops, slab_bytes=None):
    size, first, last, off = (np.asarray(a) for a in (size, first, last, off))
    top = int((off + size).max()) if size.size else 0
    slab = torch.empty(max(slab_bytes if slab_bytes is not None else top, 4),
                       dtype=torch.uint8, device="cuda")
    clob, cnt = binding.probe_plan(dev(size, torch.int64), dev(first, torch.int32),
                                   dev(last, torch.int32), dev(off, torch.int64), num_ops, slab)
    return host(clob).astype(bool), int(cnt.item())


def _check(binding, size, first, last, off, num_ops):
    g, gc = _probe(binding, size, first, last, off, num_ops)
    e, ec = oracle.probe_plan(size, first, last, off, num_ops)
    bad = np.nonzero(g != e)[0]
    assert bad.size == 0, f"{bad.size} tensors differ, first at {bad[:5]}"
    assert gc == ec
    return gc


def test_hand_cases():
    binding = need_gpu()
    print("case probe hand cases", flush=True)
    assert _check(binding, [64, 128, 192], [0, 0, 0], [2, 2, 2], [0, 0, 0], 3) == 2
    assert _check(binding, [64, 64], [0, 1], [0, 1], [0, 0], 2) == 0
    assert _check(binding, [64, 64], [1, 0], [1, 0], [0, 0], 2) == 0
    assert _check(binding, [64, 64], [1, 0], [1, 1], [0, 32], 2) == 1


def test_random_plans_with_conflicts():
    binding = need_gpu()
    rng = np.random.default_rng(41)
    print("case probe random plans", flush=True)
    for _ in range(40):
        n = int(rng.integers(1, 400))
        size = 4 * rng.integers(1, 200, n)  # multiples of 4 bytes, ranges of many words
        first = rng.integers(0, 30, n)
        last = first + rng.integers(0, 10, n)
        off = 4 * rng.integers(0, 3000, n)
        _check(binding, size, first, last, off, int(last.max()) + 1)


def test_decode100k_clean_and_corrupted():
    binding = need_gpu()
    print("case probe decode100k (planned on the GPU, then 100 offsets perturbed)", flush=True)
    t = tg.decode100k()
    o, p = binding.plan_trace(dev(t.size, torch.int64), dev(t.first, torch.int32),
                              dev(t.last, torch.int32), t.num_ops)
    off = host(o)
    assert _check(binding, t.size, t.first, t.last, off, t.num_ops) == 0
    bad, chosen = tg.corrupt_offsets(t.first, t.last, off, seed=5, k=100)
    n_clob = _check(binding, t.size, t.first, t.last, bad, t.num_ops)
    assert n_clob > 0


def test_apply_plan_views_and_errors():
    binding = need_gpu()
    print("case apply_plan views, probe status codes", flush=True)
    slab, views = binding.apply_plan([0, 64, 128], [64, 64, 32], 160)
    assert [v.data_ptr() - slab.data_ptr() for v in views] == [0, 64, 128]
    assert [v.numel() for v in views] == [64, 64, 32]
    # a size that is not a multiple of 4, and a slab smaller than the plan
    for size, off, slab_bytes in (([62], [0], 64), ([64], [0], 32)):
        st = binding.new_status()
        s = torch.empty(slab_bytes, dtype=torch.uint8, device="cuda")
        binding.probe_plan(dev(np.array(size), torch.int64), dev(np.array([0]), torch.int32),
                           dev(np.array([0]), torch.int32), dev(np.array(off), torch.int64), 1, s,
                           check=False, status=st)
        assert int(st.item()) == binding.MP_EINVAL
    # empty trace
    assert _probe(binding, np.zeros(0, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32),
                  np.zeros(0, np.int64), 3)[1] == 0
