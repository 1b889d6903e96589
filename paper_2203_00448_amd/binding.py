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

MP_OK, MP_EINVAL, MP_ENOSPC, MP_EOVERFLOW, MP_EDEVICE = 0, -1, -2, -3, -4
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
               out=None, status=None, stream=None):
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
    rc = L.mp_plan_batch(_p(begin), n_traces, _p(num_ops), _p(size), _p(first), _p(last), n,
                         int(max_trace_len), int(policy), _p(offset), _p(peak), _p(lb),
                         None, 0, _p(status), _stream(stream))
    _finish(rc, status, "plan_batch", check)
    return offset, peak, lb
