"""Plain CPU oracle of greedy-by-size static memory planning.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
baseline of the benchmark import this package; the product path never does.
It wraps `libmemoplan_oracle.so` (plain single-threaded C in this directory,
no code shared with the GPU library) with numpy marshalling.

What it computes follows Levental, "Memory Planning for Deep Neural
Networks": the offline dynamic-storage-allocation problem of Section 2.3
(sizes and lifetimes known, find one arena size and an offset per tensor) solved
by greedy_by_size (Section 2.3, chosen as the planner in Section 3.2); plan
validity is the pairwise non-overlap constraint of Eq. 2.1.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmemoplan_oracle.so")
SRC_PATH = os.path.join(HERE, "memoplan_oracle.c")

OK, EINVAL, ENOSPC, EOVERFLOW = 0, -1, -2, -3
LOWEST_FIT, BEST_FIT = 0, 1


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: oracle status {status}")
        self.status = status


def build(force: bool = True) -> str:
    """Compile the oracle with the host C compiler (gcc)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                        "-o", tmp, SRC_PATH], check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=True)
        L = ctypes.CDLL(LIB_PATH)
        p = ctypes.c_void_p
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        L.mpo_check_trace.argtypes = [p, p, p, i64, i32]
        L.mpo_rank_order.argtypes = [p, p, i64, p]
        L.mpo_plan_trace.argtypes = [p, p, p, i64, i32, i32, p, p]
        L.mpo_plan_trace_w.argtypes = [p, p, p, i64, i32, i32, i32, p, p]
        L.mpo_live_bytes_profile.argtypes = [p, p, p, i64, i32, p, p]
        L.mpo_validate_plan.argtypes = [p, p, p, p, i64, p, i64, p]
        L.mpo_probe_plan.argtypes = [p, p, p, p, i64, i32, p, p]
        L.mpo_bump_plan.argtypes = [p, p, p, i64, i32, p, p]
        L.mpo_optimal_plan.argtypes = [p, p, p, i64, i32, p, p]
        L.mpo_breadth_order.argtypes = [p, p, p, i64, i32, p]
        L.mpo_plan_breadth.argtypes = [p, p, p, i64, i32, i32, p, p]
        L.mpo_dag_depth.argtypes = [p, p, p, i64, i32, p, p]
        for f in (L.mpo_check_trace, L.mpo_rank_order, L.mpo_plan_trace, L.mpo_plan_trace_w,
                  L.mpo_live_bytes_profile, L.mpo_validate_plan, L.mpo_probe_plan):
            f.restype = i32
        _lib = L
    return _lib


def _arr(x, dt):
    return np.ascontiguousarray(x, dtype=dt)


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a.size else None


def check_trace(size, first, last, num_ops: int) -> int:
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    return lib().mpo_check_trace(_ptr(s), _ptr(f), _ptr(l), s.shape[0], int(num_ops))


def rank_order(size, first) -> np.ndarray:
    s, f = _arr(size, np.int64), _arr(first, np.int32)
    out = np.empty(s.shape[0], np.int32)
    st = lib().mpo_rank_order(_ptr(s), _ptr(f), s.shape[0], _ptr(out))
    if st != OK:
        raise OracleError(st, "rank_order")
    return out


def plan_trace(size, first, last, num_ops: int, policy: int = LOWEST_FIT,
               bucket_width: int | None = None):
    """Greedy-by-size offsets and peak for one trace: returns (offset int64[n], peak)."""
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    off = np.zeros(s.shape[0], np.int64)
    peak = ctypes.c_int64(0)
    if bucket_width is None:
        st = lib().mpo_plan_trace(_ptr(s), _ptr(f), _ptr(l), s.shape[0], int(num_ops), int(policy),
                                  _ptr(off), ctypes.byref(peak))
    else:
        st = lib().mpo_plan_trace_w(_ptr(s), _ptr(f), _ptr(l), s.shape[0], int(num_ops),
                                    int(policy), int(bucket_width), _ptr(off), ctypes.byref(peak))
    if st != OK:
        raise OracleError(st, "plan_trace")
    return off, int(peak.value)


def dag_depth(size, first, last, num_ops: int):
    """Levels of greedy_by_size's dependency structure (1 + the largest level
    among the earlier-ranked tensors a tensor meets) and their maximum, the
    depth.  Returns (level int32[n], depth)."""
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    level = np.zeros(s.shape[0], np.int32)
    depth = ctypes.c_int32(0)
    st = lib().mpo_dag_depth(_ptr(s), _ptr(f), _ptr(l), s.shape[0], int(num_ops), _ptr(level),
                             ctypes.byref(depth))
    if st != OK:
        raise OracleError(st, "dag_depth")
    return level, int(depth.value)


def plan_batch(begin, num_ops, size, first, last, policy: int = LOWEST_FIT):
    """Each trace b = tensors [begin[b], begin[b+1]) planned on its own; ids are
    local to the trace.  Returns (offset int64[N], peak int64[B])."""
    begin = _arr(begin, np.int64)
    num_ops = _arr(num_ops, np.int32)
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    off = np.zeros(s.shape[0], np.int64)
    peak = np.zeros(num_ops.shape[0], np.int64)
    for b in range(num_ops.shape[0]):
        lo, hi = int(begin[b]), int(begin[b + 1])
        off[lo:hi], peak[b] = plan_trace(s[lo:hi], f[lo:hi], l[lo:hi], int(num_ops[b]), policy)
    return off, peak


def live_bytes_profile(size, first, last, num_ops: int):
    """Returns (live int64[num_ops], max_live)."""
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    live = np.zeros(int(num_ops), np.int64)
    mx = ctypes.c_int64(0)
    st = lib().mpo_live_bytes_profile(_ptr(s), _ptr(f), _ptr(l), s.shape[0], int(num_ops),
                                      _ptr(live), ctypes.byref(mx))
    if st != OK:
        raise OracleError(st, "live_bytes_profile")
    return live, int(mx.value)


def validate_plan(size, first, last, offset, capacity: int | None = None):
    """Returns (pairs int64[k, 2], exact count).  capacity=None sizes the output
    from a counting call; a smaller capacity raises OracleError(ENOSPC) when the
    count exceeds it."""
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    o = _arr(offset, np.int64)
    cnt = ctypes.c_int64(0)
    if capacity is None:
        st = lib().mpo_validate_plan(_ptr(s), _ptr(f), _ptr(l), _ptr(o), s.shape[0], None, 0,
                                     ctypes.byref(cnt))
        if st not in (OK, ENOSPC):
            raise OracleError(st, "validate_plan")
        capacity = int(cnt.value)
    pairs = np.zeros((max(capacity, 0), 2), np.int64)
    st = lib().mpo_validate_plan(_ptr(s), _ptr(f), _ptr(l), _ptr(o), s.shape[0], _ptr(pairs),
                                 int(capacity), ctypes.byref(cnt))
    if st != OK:
        raise OracleError(st, "validate_plan")
    return pairs[: int(cnt.value)], int(cnt.value)


def probe_plan(size, first, last, offset, num_ops: int):
    """Write-pattern aliasing probe of a plan (see mpo_probe_plan).  Returns
    (clobbered bool[n], count)."""
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    o = _arr(offset, np.int64)
    out = np.zeros(s.shape[0], np.uint8)
    cnt = ctypes.c_int64(0)
    st = lib().mpo_probe_plan(_ptr(s), _ptr(f), _ptr(l), _ptr(o), s.shape[0], int(num_ops),
                              _ptr(out), ctypes.byref(cnt))
    if st != OK:
        raise OracleError(st, "probe_plan")
    return out.astype(bool), int(cnt.value)


OPT_MAX_N = 12


def _offsets_call(fn, what, size, first, last, num_ops):
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    off = np.zeros(s.shape[0], np.int64)
    peak = ctypes.c_int64(0)
    st = fn(_ptr(s), _ptr(f), _ptr(l), s.shape[0], int(num_ops), _ptr(off), ctypes.byref(peak))
    if st != OK:
        raise OracleError(st, what)
    return off, int(peak.value)


def bump_plan(size, first, last, num_ops: int):
    """bump_allocation (Section 2.3): (offsets, peak = sum of sizes)."""
    return _offsets_call(lib().mpo_bump_plan, "bump_plan", size, first, last, num_ops)


def optimal_plan(size, first, last, num_ops: int):
    """The optimum of Eq. 2.1 by exhaustive search over placement orders
    (n <= OPT_MAX_N): (offsets of one optimal plan, optimal peak)."""
    return _offsets_call(lib().mpo_optimal_plan, "optimal_plan", size, first, last, num_ops)


def breadth_order(size, first, last, num_ops: int) -> np.ndarray:
    """Greedy by Breadth placement order (Section 6, Pisarchyk et al.)."""
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    out = np.zeros(s.shape[0], np.int32)
    st = lib().mpo_breadth_order(_ptr(s), _ptr(f), _ptr(l), s.shape[0], int(num_ops), _ptr(out))
    if st != OK:
        raise OracleError(st, "breadth_order")
    return out


def plan_breadth(size, first, last, num_ops: int, policy: int = LOWEST_FIT):
    """Greedy by Breadth offsets and peak."""
    s, f, l = _arr(size, np.int64), _arr(first, np.int32), _arr(last, np.int32)
    off = np.zeros(s.shape[0], np.int64)
    peak = ctypes.c_int64(0)
    st = lib().mpo_plan_breadth(_ptr(s), _ptr(f), _ptr(l), s.shape[0], int(num_ops), int(policy),
                                _ptr(off), ctypes.byref(peak))
    if st != OK:
        raise OracleError(st, "plan_breadth")
    return off, int(peak.value)
