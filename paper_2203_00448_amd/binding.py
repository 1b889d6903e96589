"""Python binding of libmemoplan.so (ctypes): argument marshalling only.

Every computation happens in the HIP kernels behind the C ABI declared in
include/memoplan.h.  torch is used for device memory and the current stream.
If the library is missing the calls raise; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmemoplan.so")
# test build (MP_DEBUG_WAIT): mp_plan_trace honours MEMOPLAN_DEBUG_WAIT
DBG_WAIT_LIB_PATH = os.path.join(PKG, "libmemoplan_dbgwait.so")

MP_OK, MP_EINVAL, MP_ENOSPC, MP_EOVERFLOW, MP_EDEVICE = 0, -1, -2, -3, -4
OP_LIVE_BYTES, OP_VALIDATE, OP_PLAN_TRACE, OP_VALIDATE_BATCH, OP_PLAN_BATCH = 1, 2, 3, 4, 5
OP_PROBE = 6
OP_BUMP = 7
OPT_MAX_N = 12
BREADTH_MAX_TRACE_LEN = 2048
HINT_SORTED_FIRST = 1
LOWEST_FIT, BEST_FIT = 0, 1
BATCH_MAX_TRACE_LEN = 4096

_lib = None


class PlanError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


def load_library(path: str = LIB_PATH):
    """Load libmemoplan.so (built by paper_2203_00448_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libmemoplan.so not built ({path}); run paper_2203_00448_amd/build.py")
    L = ctypes.CDLL(path)
    p, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    L.mp_status_string.argtypes = [i32]
    L.mp_status_string.restype = ctypes.c_char_p
    L.mp_status_reset.argtypes = [p, p]
    L.mp_status_reset.restype = i32
    L.mp_batch_pair_capacity.argtypes = [i64]
    L.mp_batch_pair_capacity.restype = i64
    L.mp_plan_batch.argtypes = [p, i64, p, p, p, p, i64, i64, i32, p, p, p, p, sz, p, p]
    L.mp_plan_batch.restype = i32
    L.mp_workspace_size.argtypes = [i32, i64, i64, i64]
    L.mp_workspace_size.restype = sz
    L.mp_workspace_bytes.argtypes = [i32, i64, i64, i64]
    L.mp_workspace_bytes.restype = sz
    L.mp_live_bytes_profile.argtypes = [p, p, p, i64, i32, p, p, p, sz, p, p]
    L.mp_live_bytes_profile.restype = i32
    L.mp_live_bytes_profile_noalloc.argtypes = [p, p, p, i64, i32, p, p, p, p]
    L.mp_live_bytes_profile_noalloc.restype = i32
    L.mp_validate_plan.argtypes = [p, p, p, p, i64, p, i64, p, i32, p, sz, p, p]
    L.mp_validate_plan.restype = i32
    L.mp_validate_batch.argtypes = [p, i64, p, p, p, p, i64, i64, p, i64, p, i32, p, sz, p, p]
    L.mp_validate_batch.restype = i32
    L.mp_plan_trace.argtypes = [p, p, p, i64, i32, i32, p, p, p, sz, p, p]
    L.mp_plan_trace.restype = i32
    L.mp_probe_plan.argtypes = [p, p, p, p, i64, i32, p, sz, p, p, p, sz, p, p]
    L.mp_probe_plan.restype = i32
    L.mp_bump_plan.argtypes = [p, i64, p, p, p, i64, i32, p, p, p, sz, p, p]
    L.mp_bump_plan.restype = i32
    L.mp_optimal_batch.argtypes = [p, i64, p, p, p, p, i64, p, p, p, p]
    L.mp_optimal_batch.restype = i32
    L.mp_plan_breadth_batch.argtypes = [p, i64, p, p, p, p, i64, i32, p, p, p, p]
    L.mp_plan_breadth_batch.restype = i32
    _lib = L
    return L


def status_string(status: int) -> str:
    return load_library().mp_status_string(int(status)).decode()


def _dev(t: torch.Tensor, dtype, name):
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t.contiguous()


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() else None


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def new_status(device="cuda", stream=None) -> torch.Tensor:
    """A device status word reset to MP_OK on the stream."""
    st = torch.empty(1, dtype=torch.int32, device=device)
    reset_status(st, stream)
    return st


def reset_status(status: torch.Tensor, stream=None):
    rc = load_library().mp_status_reset(_p(status), _stream(stream))
    if rc != MP_OK:
        raise PlanError(rc, "status_reset")


def _finish(rc: int, status: torch.Tensor, what: str, check: bool):
    if rc != MP_OK:
        raise PlanError(rc, what)
    if check:
        st = int(status.item())  # synchronises with the stream
        if st != MP_OK:
            raise PlanError(st, what)


def batch_pair_capacity(max_trace_len: int) -> int:
    return int(load_library().mp_batch_pair_capacity(int(max_trace_len)))


def plan_batch(begin, num_ops, size, first, last, *, max_trace_len: int | None = None,
               policy: int = LOWEST_FIT, with_lb: bool = True, check: bool = True,
               out=None, status=None, stream=None, workspace=None):
    """Greedy-by-size plans of many traces (mp_plan_batch).

    begin int64[B+1], num_ops int32[B], size int64[N], first/last int32[N], all
    on the GPU.  Returns (offset int64[N], peak int64[B], lb int64[B] or None).
    The device status word is sticky (atomic minimum over calls): without a
    `status` argument a fresh one is made.  With check=True the call waits for
    the stream and raises PlanError on a device status; with check=False the
    caller inspects `status` later."""
    L = load_library()
    begin = _dev(begin, torch.int64, "begin")
    num_ops = _dev(num_ops, torch.int32, "num_ops")
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    n_traces = num_ops.numel()
    n = size.numel()
    if begin.numel() != n_traces + 1 or first.numel() != n or last.numel() != n:
        raise ValueError("inconsistent array lengths")
    if max_trace_len is None:
        max_trace_len = int((begin[1:] - begin[:-1]).max().item()) if n_traces else 0
    dev = size.device
    if out is None:
        offset = torch.empty(n, dtype=torch.int64, device=dev)
        peak = torch.empty(n_traces, dtype=torch.int64, device=dev)
        lb = torch.empty(n_traces, dtype=torch.int64, device=dev) if with_lb else None
    else:
        offset, peak, lb = out
    if status is None:
        status = new_status(dev, stream)
    ws, need = _workspace(OP_PLAN_BATCH, dev, n, n_traces, 0, workspace)
    rc = L.mp_plan_batch(_p(begin), n_traces, _p(num_ops), _p(size), _p(first), _p(last), n,
                         int(max_trace_len), int(policy), _p(offset), _p(peak), _p(lb),
                         _p(ws), need, _p(status), _stream(stream))
    _finish(rc, status, "plan_batch", check)
    return offset, peak, lb


def workspace_size(op: int, n_tensors: int = 0, num_ops: int = 0, capacity: int = 0) -> int:
    """mp_workspace_size: bytes of workspace for `op`; for MP_OP_PLAN_BATCH
    num_ops carries the number of traces, for the validation and probe ops
    capacity the output capacity."""
    return int(load_library().mp_workspace_size(int(op), int(n_tensors), int(num_ops),
                                                 int(capacity)))


def workspace_bytes(op: int, n_tensors: int = 0, max_num_ops: int = 0, n_traces: int = 1) -> int:
    """mp_workspace_bytes: bytes of workspace for `op` from the tensor count,
    the largest op count and the number of traces."""
    return int(load_library().mp_workspace_bytes(int(op), int(n_tensors), int(max_num_ops),
                                                  int(n_traces)))


def _workspace(op, dev, n_tensors=0, num_ops=0, capacity=0, workspace=None):
    need = workspace_size(op, n_tensors, num_ops, capacity)
    if workspace is not None:
        if workspace.numel() * workspace.element_size() < need:
            raise ValueError(f"workspace needs {need} bytes")
        return workspace, need
    return torch.empty(max(need, 1), dtype=torch.uint8, device=dev), need


def live_bytes_profile(size, first, last, num_ops: int, *, check: bool = True, out=None,
                       status=None, workspace=None, stream=None):
    """Per-op live bytes of one trace (mp_live_bytes_profile).
    Returns (live int64[num_ops], max_live int64[1]) on the GPU."""
    L = load_library()
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    n = size.numel()
    dev = size.device
    if out is None:
        live = torch.empty(int(num_ops), dtype=torch.int64, device=dev)
        mx = torch.empty(1, dtype=torch.int64, device=dev)
    else:
        live, mx = out
    ws, need = _workspace(OP_LIVE_BYTES, dev, n, num_ops, 0, workspace)
    if status is None:
        status = new_status(dev, stream)
    rc = L.mp_live_bytes_profile(_p(size), _p(first), _p(last), n, int(num_ops), _p(live), _p(mx),
                                 _p(ws), need, _p(status), _stream(stream))
    _finish(rc, status, "live_bytes_profile", check)
    return live, mx


LIVE_NOALLOC_MAX_OPS = 1 << 24


def live_bytes_profile_noalloc(size, first, last, num_ops: int, *, out, check: bool = True,
                               status=None, stream=None):
    """mp_live_bytes_profile_noalloc: the per-op live bytes without a workspace
    (the library's static device scratch; calls on one GPU must not overlap).
    `out` = (live int64[num_ops], max_live int64[1]) preallocated by the caller."""
    L = load_library()
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    live, mx = out
    if status is None:
        status = new_status(size.device, stream)
    rc = L.mp_live_bytes_profile_noalloc(_p(size), _p(first), _p(last), size.numel(),
                                         int(num_ops), _p(live), _p(mx), _p(status),
                                         _stream(stream))
    _finish(rc, status, "live_bytes_profile_noalloc", check)
    return live, mx


def _validate(begin, size, first, last, offset, capacity, check, status, workspace, stream,
              out=None, assume_sorted=False, max_trace_len=0):
    L = load_library()
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    offset = _dev(offset, torch.int64, "offset")
    n = size.numel()
    dev = size.device
    if capacity is None:
        capacity = 1 << 20
    if out is None:
        pairs = torch.empty((int(capacity), 2), dtype=torch.int64, device=dev)
        count = torch.empty(1, dtype=torch.int64, device=dev)
    else:
        pairs, count = out
    if begin is None:
        ws, need = _workspace(OP_VALIDATE, dev, n, 0, capacity, workspace)
    else:
        begin = _dev(begin, torch.int64, "begin")
        ws, need = _workspace(OP_VALIDATE_BATCH, dev, n, begin.numel() - 1, capacity, workspace)
    if status is None:
        status = new_status(dev, stream)
    hints = HINT_SORTED_FIRST if assume_sorted else 0
    if begin is None:
        rc = L.mp_validate_plan(_p(size), _p(first), _p(last), _p(offset), n, _p(pairs),
                                int(capacity), _p(count), hints, _p(ws), need, _p(status),
                                _stream(stream))
    else:
        rc = L.mp_validate_batch(_p(begin), begin.numel() - 1, _p(size), _p(first), _p(last),
                                 _p(offset), n, int(max_trace_len), _p(pairs), int(capacity),
                                 _p(count), hints, _p(ws), need, _p(status), _stream(stream))
    if rc != MP_OK:
        raise PlanError(rc, "validate")
    if check:
        st = int(status.item())
        if st not in (MP_OK, MP_ENOSPC):
            raise PlanError(st, "validate")
        k = int(count.item())
        return pairs[: min(k, int(capacity))], k, st
    return pairs, count, status


def validate_plan(size, first, last, offset, *, capacity: int | None = None, check: bool = True,
                  status=None, workspace=None, stream=None, out=None, assume_sorted=False):
    """All lifetime-intersecting pairs whose byte ranges overlap (mp_validate_plan).
    With check=True returns (pairs[k, 2] lexicographic, exact count k, status);
    status is MP_ENOSPC when k exceeds capacity (only capacity pairs returned)."""
    return _validate(None, size, first, last, offset, capacity, check, status, workspace, stream,
                     out, assume_sorted)


def validate_batch(begin, size, first, last, offset, *, capacity: int | None = None,
                   check: bool = True, status=None, workspace=None, stream=None, out=None,
                   assume_sorted=False, max_trace_len: int = 0):
    """mp_validate_batch: like validate_plan over the traces begin[b]..begin[b+1].
    With assume_sorted and a nonzero max_trace_len (a bound on every trace's
    length, at most BATCH_MAX_TRACE_LEN) each trace is checked in one
    workgroup."""
    return _validate(begin, size, first, last, offset, capacity, check, status, workspace, stream,
                     out, assume_sorted, max_trace_len)


def plan_trace(size, first, last, num_ops: int, *, policy: int = LOWEST_FIT, check: bool = True,
               out=None, status=None, workspace=None, stream=None):
    """Greedy-by-size plan of one trace on the whole device (mp_plan_trace).
    Returns (offset int64[n], peak int64[1]) on the GPU."""
    L = load_library()
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    n = size.numel()
    dev = size.device
    if out is None:
        offset = torch.empty(n, dtype=torch.int64, device=dev)
        peak = torch.empty(1, dtype=torch.int64, device=dev)
    else:
        offset, peak = out
    ws, need = _workspace(OP_PLAN_TRACE, dev, n, num_ops, 0, workspace)
    if status is None:
        status = new_status(dev, stream)
    rc = L.mp_plan_trace(_p(size), _p(first), _p(last), n, int(num_ops), int(policy), _p(offset),
                         _p(peak), _p(ws), need, _p(status), _stream(stream))
    _finish(rc, status, "plan_trace", check)
    return offset, peak


def apply_plan(offset, size, peak: int, device="cuda"):
    """The plan applied as in Section 3.3: one slab of `peak` bytes and every
    tensor a byte view at its offset (offset, size: host integer sequences).
    Returns (slab uint8[peak], views); allocation and views are torch's."""
    slab = torch.empty(max(int(peak), 4), dtype=torch.uint8, device=device)
    views = [slab.narrow(0, int(o), int(s)) for o, s in zip(offset, size)]
    return slab, views


def probe_plan(size, first, last, offset, num_ops: int, slab: torch.Tensor, *,
               check: bool = True, out=None, status=None, workspace=None, stream=None,
               capacity: int = 0):
    """Write-pattern aliasing probe of a plan over `slab` (mp_probe_plan).
    `capacity` sizes a new workspace: the (tensor, 256-byte tile) pairs the
    tiled replay holds (0: the library's default); a plan with more pairs is
    replayed op by op.  Returns (clobbered uint8[n], n_clobbered int64[1])."""
    L = load_library()
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    offset = _dev(offset, torch.int64, "offset")
    n = size.numel()
    dev = size.device
    if slab.device != dev or not slab.is_contiguous():
        raise ValueError("slab must be a contiguous tensor on the device of the trace")
    if out is None:
        clob = torch.empty(max(n, 1), dtype=torch.uint8, device=dev)[:n]
        cnt = torch.empty(1, dtype=torch.int64, device=dev)
    else:
        clob, cnt = out
    # the library takes the largest capacity the workspace holds (MP_EINVAL
    # if it is too small even for the op-by-op replay)
    ws = workspace if workspace is not None else _workspace(OP_PROBE, dev, n, num_ops,
                                                            capacity)[0]
    if status is None:
        status = new_status(dev, stream)
    rc = L.mp_probe_plan(_p(size), _p(first), _p(last), _p(offset), n, int(num_ops), _p(slab),
                         slab.numel() * slab.element_size(), _p(clob), _p(cnt), _p(ws),
                         ws.numel() * ws.element_size(), _p(status), _stream(stream))
    _finish(rc, status, "probe_plan", check)
    return clob, cnt


def bump_plan(size, first, last, num_ops: int, *, begin=None, check: bool = True, out=None,
              status=None, workspace=None, stream=None):
    """bump_allocation (mp_bump_plan): offsets at the running sum of sizes in
    allocation order (first op, then id).  One trace, or many with `begin`
    (num_ops then bounds every trace's op count).  Returns (offset int64[n],
    peak int64[traces])."""
    L = load_library()
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    n = size.numel()
    if first.numel() != n or last.numel() != n:
        raise ValueError("inconsistent array lengths")
    dev = size.device
    n_traces = 1
    if begin is not None:
        begin = _dev(begin, torch.int64, "begin")
        n_traces = begin.numel() - 1
        if n_traces < 0:
            raise ValueError("begin needs at least one entry")
    if out is None:
        offset = torch.empty(max(n, 1), dtype=torch.int64, device=dev)[:n]
        peak = torch.empty(max(n_traces, 1), dtype=torch.int64, device=dev)[:n_traces]
    else:
        offset, peak = out
    if status is None:
        status = new_status(dev, stream)
    ws, need = _workspace(OP_BUMP, dev, n, 0, 0, workspace)
    rc = L.mp_bump_plan(_p(begin) if begin is not None else None, n_traces, _p(size), _p(first),
                        _p(last), n, int(num_ops), _p(offset), _p(peak), _p(ws), need,
                        _p(status), _stream(stream))
    _finish(rc, status, "bump_plan", check)
    return offset, peak


def optimal_batch(begin, num_ops, size, first, last, *, check: bool = True, out=None,
                  status=None, stream=None):
    """The optimum of Eq. 2.1 for tiny traces (at most OPT_MAX_N tensors each)
    by exhaustive search (mp_optimal_batch).  Returns (offset int64[N] of one
    optimal plan per trace, peak int64[B] = the optimum)."""
    L = load_library()
    begin = _dev(begin, torch.int64, "begin")
    num_ops = _dev(num_ops, torch.int32, "num_ops")
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    n_traces, n = num_ops.numel(), size.numel()
    if begin.numel() != n_traces + 1 or first.numel() != n or last.numel() != n:
        raise ValueError("inconsistent array lengths")
    dev = size.device
    if out is None:
        offset = torch.empty(max(n, 1), dtype=torch.int64, device=dev)[:n]
        peak = torch.empty(max(n_traces, 1), dtype=torch.int64, device=dev)[:n_traces]
    else:
        offset, peak = out
    if status is None:
        status = new_status(dev, stream)
    rc = L.mp_optimal_batch(_p(begin), n_traces, _p(num_ops), _p(size), _p(first), _p(last), n,
                            _p(offset), _p(peak), _p(status), _stream(stream))
    _finish(rc, status, "optimal_batch", check)
    return offset, peak


def plan_breadth_batch(begin, num_ops, size, first, last, *, policy: int = LOWEST_FIT,
                       check: bool = True, out=None, status=None, stream=None):
    """Greedy by Breadth plans of many traces (mp_plan_breadth_batch), each at
    most BREADTH_MAX_TRACE_LEN tensors.  Returns (offset int64[N], peak int64[B])."""
    L = load_library()
    begin = _dev(begin, torch.int64, "begin")
    num_ops = _dev(num_ops, torch.int32, "num_ops")
    size = _dev(size, torch.int64, "size")
    first = _dev(first, torch.int32, "first")
    last = _dev(last, torch.int32, "last")
    n_traces, n = num_ops.numel(), size.numel()
    if begin.numel() != n_traces + 1 or first.numel() != n or last.numel() != n:
        raise ValueError("inconsistent array lengths")
    dev = size.device
    if out is None:
        offset = torch.empty(max(n, 1), dtype=torch.int64, device=dev)[:n]
        peak = torch.empty(max(n_traces, 1), dtype=torch.int64, device=dev)[:n_traces]
    else:
        offset, peak = out
    if status is None:
        status = new_status(dev, stream)
    rc = L.mp_plan_breadth_batch(_p(begin), n_traces, _p(num_ops), _p(size), _p(first), _p(last),
                                 n, int(policy), _p(offset), _p(peak), _p(status), _stream(stream))
    _finish(rc, status, "plan_breadth_batch", check)
    return offset, peak
