"""Parity of the plan-application probe on the GPU with the CPU oracle.

The plan applied as in Section 3.3 (one slab, every tensor a view at its
offset, Listing 5) and exercised by replaying the ops: each tensor writes
id + 1 into its words at its first op (the larger value kept), checks them at
its last op and clears them.  Which tensors find a foreign word is integer
work and does not depend on the order of one op's writers, so the GPU result
must equal the oracle's bit for bit, on both of the library's paths: the
replay split into 256-byte tiles (one wave each) and the op-by-op replay
that takes over when the workspace cannot hold the plan's (tensor, tile)
pairs.  The workspace starts with the path flags (int32 words: bad input,
tiled kernels skipped, op-by-op replay run), which the tests read to make
sure each path really ran.
"""
import numpy as np
import pytest

import oracle
from gpu_util import dev, host, need_gpu, torch
from paper_2203_00448_amd import tracegen as tg

pytestmark = pytest.mark.gpu
TILED, OPS = 0, 1


def _pairs(size, off):
    w0, w1 = np.asarray(off) // 4, (np.asarray(off) + np.asarray(size)) // 4
    return int(((((w1 - 1) >> 6) - (w0 >> 6)) + 1).sum())


def _probe(binding, size, first, last, off, num_ops, capacity=0):
    size, first, last, off = (np.asarray(a) for a in (size, first, last, off))
    top = int((off + size).max()) if size.size else 0
    slab = torch.empty(max(top, 4), dtype=torch.uint8, device="cuda")
    ws = torch.empty(binding.workspace_size(binding.OP_PROBE, size.size, num_ops, capacity),
                     dtype=torch.uint8, device="cuda")
    clob, cnt = binding.probe_plan(dev(size, torch.int64), dev(first, torch.int32),
                                   dev(last, torch.int32), dev(off, torch.int64), num_ops, slab,
                                   workspace=ws)
    flags = host(ws[:12].view(torch.int32))
    return host(clob).astype(bool), int(cnt.item()), int(flags[2])


def _check(binding, size, first, last, off, num_ops, capacity=0, path=None):
    g, gc, ran_ops = _probe(binding, size, first, last, off, num_ops, capacity)
    e, ec = oracle.probe_plan(size, first, last, off, num_ops)
    bad = np.nonzero(g != e)[0]
    assert bad.size == 0, f"{bad.size} tensors differ, first at {bad[:5]}"
    assert gc == ec
    if path is not None:
        assert ran_ops == path
    return gc


def _both(binding, size, first, last, off, num_ops):
    """Tiled with the default capacity, op by op with a capacity of one pair."""
    c = _check(binding, size, first, last, off, num_ops, path=TILED)
    many = _pairs(size, off) > 1
    assert _check(binding, size, first, last, off, num_ops, capacity=1,
                  path=OPS if many else TILED) == c
    return c


def test_hand_cases():
    binding = need_gpu()
    print("case probe hand cases, both paths", flush=True)
    assert _both(binding, [64, 128, 192], [0, 0, 0], [2, 2, 2], [0, 0, 0], 3) == 2
    assert _both(binding, [64, 64], [0, 1], [0, 1], [0, 0], 2) == 0
    assert _both(binding, [64, 64], [1, 0], [1, 0], [0, 0], 2) == 0
    assert _both(binding, [64, 64], [1, 0], [1, 1], [0, 32], 2) == 1
    # ranges crossing tile boundaries (256 bytes), overlaps inside one tile
    assert _both(binding, [512, 260, 8], [0, 1, 1], [1, 2, 1], [0, 252, 500], 3) == 2


def test_random_plans_with_conflicts():
    binding = need_gpu()
    rng = np.random.default_rng(41)
    print("case probe random plans, both paths", flush=True)
    for _ in range(40):
        n = int(rng.integers(1, 400))
        size = 4 * rng.integers(1, 200, n)  # multiples of 4 bytes, ranges of many words
        first = rng.integers(0, 30, n)
        last = first + rng.integers(0, 10, n)
        off = 4 * rng.integers(0, 3000, n)
        _both(binding, size, first, last, off, int(last.max()) + 1)


def test_capacity_boundary():
    binding = need_gpu()
    rng = np.random.default_rng(43)
    print("case probe capacity: exactly the pairs (tiled), half of them (op by op)", flush=True)
    n = 3000
    size = 4 * rng.integers(1, 400, n)
    first = rng.integers(0, 200, n)
    last = first + rng.integers(0, 20, n)
    off = 4 * rng.integers(0, 20000, n)
    p = _pairs(size, off)
    assert p > 2000
    num_ops = int(last.max()) + 1
    c = _check(binding, size, first, last, off, num_ops, capacity=p, path=TILED)
    assert _check(binding, size, first, last, off, num_ops, capacity=p // 2, path=OPS) == c


def test_heavy_tensors_fall_back():
    binding = need_gpu()
    print("case probe 4 tensors of 8 MiB (more pairs than the default capacity)", flush=True)
    mb8 = 8 << 20
    size = np.full(4, mb8, np.int64)
    first, last = np.array([0, 1, 1, 2]), np.array([1, 2, 3, 3])
    off = np.array([0, mb8, 0, 2 * mb8 - 4096], np.int64)  # 0/1 overlap at op 1, 1/3 at op 2
    assert _pairs(size, off) > 16 * 4 + 65536
    assert _check(binding, size, first, last, off, 4, path=OPS) > 0


def test_decode100k_clean_and_corrupted():
    binding = need_gpu()
    print("case probe decode100k (planned on the GPU, then 100 offsets perturbed)", flush=True)
    t = tg.decode100k()
    o, p = binding.plan_trace(dev(t.size, torch.int64), dev(t.first, torch.int32),
                              dev(t.last, torch.int32), t.num_ops)
    off = host(o)
    assert _check(binding, t.size, t.first, t.last, off, t.num_ops, path=TILED) == 0
    bad, chosen = tg.corrupt_offsets(t.first, t.last, off, seed=5, k=100)
    n_clob = _check(binding, t.size, t.first, t.last, bad, t.num_ops, path=TILED)
    assert n_clob > 0
    assert _check(binding, t.size, t.first, t.last, bad, t.num_ops, capacity=1, path=OPS) == n_clob


def test_apply_plan_views_and_errors():
    binding = need_gpu()
    print("case apply_plan views, probe status codes", flush=True)
    slab, views = binding.apply_plan([0, 64, 128], [64, 64, 32], 160)
    assert [v.data_ptr() - slab.data_ptr() for v in views] == [0, 64, 128]
    assert [v.numel() for v in views] == [64, 64, 32]
    # a size that is not a multiple of 4, a slab smaller than the plan, a
    # last op past the trace
    for size, off, slab_bytes, last in (([62], [0], 64, 0), ([64], [0], 32, 0),
                                        ([64], [0], 64, 1)):
        st = binding.new_status()
        s = torch.empty(slab_bytes, dtype=torch.uint8, device="cuda")
        binding.probe_plan(dev(np.array(size), torch.int64), dev(np.array([0]), torch.int32),
                           dev(np.array([last]), torch.int32), dev(np.array(off), torch.int64),
                           1, s, check=False, status=st)
        assert int(st.item()) == binding.MP_EINVAL
    # empty trace
    assert _probe(binding, np.zeros(0, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32),
                  np.zeros(0, np.int64), 3)[1] == 0


def test_views_replay_chain256():
    """The slab and its views used as execution would use them: ops in order,
    each tensor written through its view at its first op and checked at its
    last -- a valid GPU plan keeps every view intact, a shifted view does not."""
    binding = need_gpu()
    print("case views replay, chain256 planned on the GPU", flush=True)
    t = tg.chain256()
    o, p = binding.plan_trace(dev(t.size, torch.int64), dev(t.first, torch.int32),
                              dev(t.last, torch.int32), t.num_ops)
    off = host(o)

    def replay(offsets):
        slab, views = binding.apply_plan(offsets, t.size, int((offsets + t.size).max()))
        slab.zero_()
        bad = []
        for op in range(t.num_ops):
            for i in np.nonzero(t.first == op)[0]:
                views[i].fill_(int(i) % 251 + 1)
            for i in np.nonzero(t.last == op)[0]:
                if not bool((views[i] == int(i) % 251 + 1).all().item()):
                    bad.append(int(i))
        return bad

    assert replay(off) == []
    # tensor 1 moved onto tensor 0's bytes: their lifetimes meet, one is hit
    moved = off.copy()
    assert t.first[1] <= t.last[0]
    moved[1] = off[0]
    assert replay(moved)


def test_sparse_plan_in_a_large_slab():
    binding = need_gpu()
    print("case probe: 64 tensors spread over 256 MiB (a million mostly empty tiles)", flush=True)
    rng = np.random.default_rng(44)
    n = 64
    size = 4 * rng.integers(1, 50000, n)
    first = rng.integers(0, 40, n)
    last = first + rng.integers(0, 6, n)
    off = (4 << 20) * rng.integers(0, 64, n) + 4 * rng.integers(0, 1000, n)  # some collide
    num_ops = int(last.max()) + 1
    c = _check(binding, size, first, last, off, num_ops, path=TILED)
    assert _check(binding, size, first, last, off, num_ops, capacity=1, path=OPS) == c
