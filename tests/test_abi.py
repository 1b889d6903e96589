"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function the public header declares, and rejects bad host arguments
before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "memoplan.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mp_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2203_00448_amd import binding
    return binding.load_library()


def test_header_declares_entry_points():
    names = declared_functions()
    for required in ("mp_plan_batch", "mp_status_string"):
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4):
        assert lib.mp_status_string(code)
    assert lib.mp_status_string(0) == b"ok"


def test_plan_batch_host_checks(lib):
    from paper_2203_00448_amd import binding as b
    dummy = ctypes.c_void_p(16)  # never dereferenced: every call below fails a host check
    st = dummy
    # negative counts
    assert lib.mp_plan_batch(dummy, -1, dummy, dummy, dummy, dummy, 0, 10, 0, dummy, dummy, None,
                             None, 0, st, None) == b.MP_EINVAL
    assert lib.mp_plan_batch(dummy, 1, dummy, dummy, dummy, dummy, -5, 10, 0, dummy, dummy, None,
                             None, 0, st, None) == b.MP_EINVAL
    # unknown policy
    assert lib.mp_plan_batch(dummy, 1, dummy, dummy, dummy, dummy, 4, 10, 7, dummy, dummy, None,
                             None, 0, st, None) == b.MP_EINVAL
    # max_trace_len out of range
    assert lib.mp_plan_batch(dummy, 1, dummy, dummy, dummy, dummy, 4, 5000, 0, dummy, dummy, None,
                             None, 0, st, None) == b.MP_EINVAL
    # missing status word / arrays
    assert lib.mp_plan_batch(dummy, 1, dummy, dummy, dummy, dummy, 4, 10, 0, dummy, dummy, None,
                             None, 0, None, None) == b.MP_EINVAL
    assert lib.mp_plan_batch(dummy, 1, dummy, None, dummy, dummy, 4, 10, 0, dummy, dummy, None,
                             None, 0, st, None) == b.MP_EINVAL
    assert lib.mp_plan_batch(None, 1, dummy, dummy, dummy, dummy, 4, 10, 0, dummy, dummy, None,
                             None, 0, st, None) == b.MP_EINVAL
    # missing or short workspace (24 bytes per tensor and 64 per trace at least)
    need = lib.mp_workspace_bytes(b.OP_PLAN_BATCH, 4, 0, 1)
    assert need >= 24 * 4 + 64
    assert lib.mp_plan_batch(dummy, 1, dummy, dummy, dummy, dummy, 4, 10, 0, dummy, dummy, None,
                             None, need, st, None) == b.MP_EINVAL
    assert lib.mp_plan_batch(dummy, 1, dummy, dummy, dummy, dummy, 4, 10, 0, dummy, dummy, None,
                             dummy, need - 1, st, None) == b.MP_EINVAL


def test_pair_capacity(lib):
    from paper_2203_00448_amd import binding as b
    assert lib.mp_batch_pair_capacity(-1) == -1
    assert lib.mp_batch_pair_capacity(4097) == -1
    assert lib.mp_batch_pair_capacity(2000) >= 12000   # the 2000-tensor traces need ~11K
    assert lib.mp_batch_pair_capacity(4096) > 0
    assert lib.mp_batch_pair_capacity(100) >= 100 * 99 // 2   # short traces: every pair
    # the batched planner's workspace: 24 bytes per tensor (the general path's
    # two offset-sorted lists, or the position permutation) + 64 per trace
    assert lib.mp_workspace_size(b.OP_PLAN_BATCH, 2048000, 1024, 0) >= 24 * 2048000 + 64 * 1024
    assert lib.mp_workspace_bytes(b.OP_PLAN_BATCH, 2048000, 0, 1024) == lib.mp_workspace_size(
        b.OP_PLAN_BATCH, 2048000, 1024, 0)
    assert lib.mp_workspace_size(b.OP_PLAN_BATCH, -1, 1, 0) == 0


def test_workspace_bytes_query(lib):
    """mp_workspace_bytes(op, n_tensors, max_num_ops, n_traces) agrees with the
    capacity-explicit query for every op (validation at capacity n_tensors)."""
    from paper_2203_00448_amd import binding as b
    wb, ws = lib.mp_workspace_bytes, lib.mp_workspace_size
    assert wb(b.OP_LIVE_BYTES, 100, 4000, 1) == ws(b.OP_LIVE_BYTES, 100, 4000, 0) > 0
    assert wb(b.OP_VALIDATE, 1000, 0, 1) == ws(b.OP_VALIDATE, 1000, 0, 1000) > 0
    assert wb(b.OP_VALIDATE_BATCH, 1000, 0, 7) == ws(b.OP_VALIDATE_BATCH, 1000, 7, 1000) > 0
    assert wb(b.OP_PLAN_TRACE, 5000, 100, 1) == ws(b.OP_PLAN_TRACE, 5000, 100, 0) > 0
    assert wb(b.OP_BUMP, 5000, 0, 1) == ws(b.OP_BUMP, 5000, 0, 0) > 0
    assert wb(b.OP_PROBE, 5000, 100, 1) == ws(b.OP_PROBE, 5000, 100, 0) > 0
    for bad in ((99, 10, 10, 1), (b.OP_PLAN_BATCH, -1, 0, 1), (b.OP_PLAN_BATCH, 10, 0, -1),
                (b.OP_LIVE_BYTES, 10, -5, 1), (b.OP_PLAN_TRACE, 1 << 30, 0, 1)):
        assert wb(*bad) == 0, bad


def test_other_host_checks(lib):
    from paper_2203_00448_amd import binding as b
    d = ctypes.c_void_p(16)
    assert lib.mp_status_reset(None, None) == b.MP_EINVAL
    # plan_trace: too many tensors, bad policy, short workspace
    assert lib.mp_plan_trace(d, d, d, 1 << 30, 10, 0, d, d, d, 1 << 40, d, None) == b.MP_EINVAL
    assert lib.mp_plan_trace(d, d, d, 10, 10, 3, d, d, d, 1 << 40, d, None) == b.MP_EINVAL
    assert lib.mp_plan_trace(d, d, d, 10, 10, 0, d, d, d, 1, d, None) == b.MP_EINVAL
    # validation: unknown hint bits, negative capacity, short workspace
    assert lib.mp_validate_plan(d, d, d, d, 10, d, 4, d, 2, d, 1 << 40, d, None) == b.MP_EINVAL
    assert lib.mp_validate_plan(d, d, d, d, 10, d, -1, d, 0, d, 1 << 40, d, None) == b.MP_EINVAL
    assert lib.mp_validate_plan(d, d, d, d, 10, d, 4, d, 0, d, 8, d, None) == b.MP_EINVAL
    assert lib.mp_validate_batch(None, 1, d, d, d, d, 10, 0, d, 4, d, 0, d, 1 << 40, d, None) == b.MP_EINVAL
    # batch validation: trace bound beyond the per-workgroup limit, short workspace
    assert lib.mp_validate_batch(d, 1, d, d, d, d, 10, b.BATCH_MAX_TRACE_LEN + 1, d, 4, d, 1, d,
                                 1 << 40, d, None) == b.MP_EINVAL
    assert lib.mp_validate_batch(d, 1, d, d, d, d, 10, -1, d, 4, d, 1, d, 1 << 40, d, None) == b.MP_EINVAL
    small = lib.mp_workspace_size(b.OP_VALIDATE_BATCH, 10, 1, 4)
    assert lib.mp_validate_batch(d, 1, d, d, d, d, 10, 16, d, 4, d, 1, d, small - 1, d, None) == b.MP_EINVAL
    # liveness: short workspace, missing outputs
    assert lib.mp_live_bytes_profile(d, d, d, 10, 10, d, d, d, 1, d, None) == b.MP_EINVAL
    assert lib.mp_live_bytes_profile(d, d, d, 10, 10, None, d, d, 1 << 40, d, None) == b.MP_EINVAL
    # workspace queries
    assert lib.mp_workspace_size(99, 10, 10, 10) == 0
    assert lib.mp_workspace_size(b.OP_VALIDATE, -1, 0, 0) == 0
    # a batch of many empty traces needs room for its per-trace counts
    assert lib.mp_workspace_size(b.OP_VALIDATE_BATCH, 0, 100000, 0) > lib.mp_workspace_size(
        b.OP_VALIDATE, 0, 0, 0)
    assert lib.mp_workspace_size(b.OP_LIVE_BYTES, 0, 100, 0) > 0
    assert lib.mp_workspace_size(b.OP_VALIDATE, 1000, 0, 100) > 0


def test_strategy_entry_points_host_checks(lib):
    from paper_2203_00448_amd import binding as b
    dummy = ctypes.c_void_p(16)  # never dereferenced: every call below fails a host check
    need = lib.mp_workspace_size(b.OP_BUMP, 10, 0, 0)
    assert need > 0
    # negative n, missing status, short workspace
    assert lib.mp_bump_plan(None, 1, dummy, dummy, dummy, -1, 4, dummy, dummy, dummy, need,
                            dummy, None) == b.MP_EINVAL
    assert lib.mp_bump_plan(None, 1, dummy, dummy, dummy, 10, 4, dummy, dummy, dummy, need,
                            None, None) == b.MP_EINVAL
    assert lib.mp_bump_plan(None, 1, dummy, dummy, dummy, 10, 4, dummy, dummy, dummy, need - 1,
                            dummy, None) == b.MP_EINVAL
    assert lib.mp_bump_plan(dummy, -3, dummy, dummy, dummy, 10, 4, dummy, dummy, dummy, need,
                            dummy, None) == b.MP_EINVAL
    # negative counts, missing arrays
    assert lib.mp_optimal_batch(dummy, -1, dummy, dummy, dummy, dummy, 4, dummy, dummy, dummy,
                                None) == b.MP_EINVAL
    assert lib.mp_optimal_batch(None, 2, dummy, dummy, dummy, dummy, 4, dummy, dummy, dummy,
                                None) == b.MP_EINVAL
    assert lib.mp_optimal_batch(dummy, 2, dummy, None, dummy, dummy, 4, dummy, dummy, dummy,
                                None) == b.MP_EINVAL
    assert lib.mp_optimal_batch(dummy, 2, dummy, dummy, dummy, dummy, 4, dummy, dummy, None,
                                None) == b.MP_EINVAL
