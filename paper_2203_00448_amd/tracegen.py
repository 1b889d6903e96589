"""Seeded synthetic allocation traces (input generation only).

The thesis profiles torchvision models to obtain, for every intermediate
tensor, a byte size and a lifetime [first_op, last_op] (Section 3.1, Table 3.1);
those traces are not available here.  This module draws stand-in traces whose
shape follows the workloads the thesis motivates (Table 1.1: CNN chains with
skip connections, decode-style traces with many short-lived tensors, ranking
models with many tensors live at once).  It contains no planning, liveness or
validation arithmetic: it only draws numbers.  Both the plain CPU oracle and
the GPU path consume exactly the arrays produced here.

Every trace is structure-of-arrays:
  size  int64[n]  bytes, > 0
  first int32[n]  op index of the first use (allocation)
  last  int32[n]  op index of the last use, first <= last < num_ops
The tensor id is the array index.

Readings of the recipes (draw order matters for reproducibility):
  r64(x)     = 64 * ceil(floor(x) / 64)       (round a real size up to 64 B)
  Geo0(p)    = rng.geometric(p) - 1           (support 0, 1, 2, ...)
  U{a..b}    = rng.integers(a, b + 1)         (inclusive integer range)
  U[a, b)    = rng.uniform(a, b) / rng.random()
"""
from __future__ import annotations

import dataclasses

import numpy as np

__all__ = [
    "Trace", "Batch", "r64", "chain256", "resnext_batch", "resnext_trace",
    "decode100k", "ranking1m", "corrupt_offsets", "random_trace",
    "CONFIG_NAMES",
]


@dataclasses.dataclass
class Trace:
    size: np.ndarray    # int64[n]
    first: np.ndarray   # int32[n]
    last: np.ndarray    # int32[n]
    num_ops: int

    @property
    def n(self) -> int:
        return int(self.size.shape[0])


@dataclasses.dataclass
class Batch:
    begin: np.ndarray    # int64[B+1], trace b owns tensors [begin[b], begin[b+1])
    num_ops: np.ndarray  # int32[B]
    size: np.ndarray     # int64[N]
    first: np.ndarray    # int32[N]
    last: np.ndarray     # int32[N]

    @property
    def n_traces(self) -> int:
        return int(self.num_ops.shape[0])

    def trace(self, b: int) -> Trace:
        lo, hi = int(self.begin[b]), int(self.begin[b + 1])
        return Trace(self.size[lo:hi], self.first[lo:hi], self.last[lo:hi],
                     int(self.num_ops[b]))


def r64(x) -> np.ndarray:
    """Round real sizes up to a multiple of 64 bytes: 64 * ceil(floor(x) / 64)."""
    fx = np.floor(np.asarray(x, dtype=np.float64)).astype(np.int64)
    return (fx + 63) // 64 * 64


def _pack(size, first, last, num_ops) -> Trace:
    return Trace(np.ascontiguousarray(size, dtype=np.int64),
                 np.ascontiguousarray(first, dtype=np.int32),
                 np.ascontiguousarray(last, dtype=np.int32), int(num_ops))


def chain256(seed: int = 1) -> Trace:
    """256 tensors over 256 ops: tensor i is born at op i and dies at
    min(255, i + 1 + Geo0(0.5)); size r64(2^u), u ~ U[10, 22) (1 KiB .. 4 MiB)."""
    rng = np.random.default_rng(seed)
    n = 256
    i = np.arange(n, dtype=np.int64)
    last = np.minimum(255, i + 1 + (rng.geometric(0.5, n) - 1))
    u = rng.uniform(10, 22, n)
    return _pack(r64(2.0 ** u), i, last, 256)


def resnext_trace(b: int, n: int = 2000) -> Trace:
    """One ResNeXt-101-like trace (seed [2, b]): n tensors over n ops, tensor i
    born at op i; 10% are skip connections living U{10..50} ops, the rest live
    U{1..3} ops; sizes log-normal (median 800 KiB, sigma 1.2) clipped to
    [4 KiB, 64 MiB], rounded up to 64 B."""
    rng = np.random.default_rng([2, b])
    i = np.arange(n, dtype=np.int64)
    skip = rng.random(n) < 0.10
    ls = rng.integers(10, 51, n)
    lc = rng.integers(1, 4, n)
    last = np.minimum(n - 1, i + np.where(skip, ls, lc))
    z = rng.standard_normal(n)
    size = r64(np.clip(np.exp(np.log(819200.0) + 1.2 * z), 4096, 2.0 ** 26))
    return _pack(size, i, last, n)


def concat(traces) -> Batch:
    traces = list(traces)
    begin = np.zeros(len(traces) + 1, dtype=np.int64)
    begin[1:] = np.cumsum([t.n for t in traces])
    cat = (lambda a, dt: np.ascontiguousarray(np.concatenate(a) if a else np.zeros(0, dt), dtype=dt))
    return Batch(begin,
                 np.asarray([t.num_ops for t in traces], dtype=np.int32),
                 cat([t.size for t in traces], np.int64),
                 cat([t.first for t in traces], np.int32),
                 cat([t.last for t in traces], np.int32))


def resnext_batch(n_traces: int = 1024, n: int = 2000) -> Batch:
    """The batched workload: traces b = 0..n_traces-1 concatenated in order."""
    return concat(resnext_trace(b, n) for b in range(n_traces))


def tiny_trace(b: int, n: int = 10) -> Trace:
    """A ResNeXt-like trace in miniature (seed [6, b]) for the exact optimum:
    n tensors over n ops, tensor i born at op i; 20% skip connections living
    U{2..max(2, n // 2)} ops, the rest U{1..2} ops; sizes as in resnext_trace
    (log-normal, median 800 KiB, sigma 1.2, clipped to [4 KiB, 64 MiB], r64)."""
    rng = np.random.default_rng([6, b])
    i = np.arange(n, dtype=np.int64)
    skip = rng.random(n) < 0.20
    ls = rng.integers(2, max(2, n // 2) + 1, n)
    lc = rng.integers(1, 3, n)
    last = np.minimum(n - 1, i + np.where(skip, ls, lc))
    z = rng.standard_normal(n)
    size = r64(np.clip(np.exp(np.log(819200.0) + 1.2 * z), 4096, 2.0 ** 26))
    return _pack(size, i, last, n)


def tiny_batch(n_traces: int = 2048, n: int = 10) -> Batch:
    """Traces b = 0..n_traces-1 of tiny_trace, concatenated."""
    return concat(tiny_trace(b, n) for b in range(n_traces))


def decode100k(seed: int = 3) -> Trace:
    """Seq2seq-decode-like trace: 4000 ops each producing 25 tensors
    (first = i // 25); lifetime Geo0(0.3) ops, and with probability 0.02 the
    tensor lives to the last op; size r64(min(256 (1-V)^(-1/1.5), 2^28))
    (Pareto alpha = 1.5 from 256 B, capped at 256 MiB)."""
    rng = np.random.default_rng(seed)
    n, t = 100_000, 4000
    i = np.arange(n, dtype=np.int64)
    first = i // 25
    last = np.minimum(t - 1, first + rng.geometric(0.3, n) - 1)
    to_end = rng.random(n) < 0.02
    last = np.where(to_end, t - 1, last)
    v = rng.random(n)
    size = r64(np.minimum(256.0 * (1.0 - v) ** (-1.0 / 1.5), 2.0 ** 28))
    return _pack(size, first, last, t)


def ranking1m(seed: int = 4) -> Trace:
    """Ranking-model-like trace: 1,000,000 tensors over 100,000 ops, ten born
    per op (first = i // 10), lifetime U{1..1000} ops, size r64(2^(6 + 10 V))
    (log-uniform in [64 B, 64 KiB])."""
    rng = np.random.default_rng(seed)
    n, t = 1_000_000, 100_000
    i = np.arange(n, dtype=np.int64)
    first = i // 10
    last = np.minimum(t - 1, first + rng.integers(1, 1001, n))
    v = rng.random(n)
    size = r64(2.0 ** (6.0 + 10.0 * v))
    return _pack(size, first, last, t)


def corrupt_offsets(first, last, offset, seed: int = 5, k: int = 100):
    """Perturb k seed-chosen offsets of a plan: S = k distinct ids; for each i in
    S (ascending) pick a tensor j outside S whose lifetime intersects i's
    (uniformly among the sorted candidates) and copy its offset to i.
    Returns (new_offsets, sorted S).  Every i in S has at least one candidate on
    the decode-like trace (its birth-op siblings)."""
    first = np.asarray(first, dtype=np.int64)
    last = np.asarray(last, dtype=np.int64)
    off = np.array(offset, dtype=np.int64, copy=True)
    n = first.shape[0]
    rng = np.random.default_rng(seed)
    chosen = np.sort(rng.choice(n, k, replace=False))
    in_s = np.zeros(n, dtype=bool)
    in_s[chosen] = True
    for i in chosen:
        cand = np.nonzero((first <= last[i]) & (first[i] <= last) & ~in_s)[0]
        if cand.size == 0:
            raise ValueError(f"tensor {i} has no lifetime neighbour outside the chosen set")
        j = cand[rng.integers(cand.size)]
        off[i] = offset[j]
    return off, chosen


def random_trace(rng: np.random.Generator, n: int, num_ops: int, *, max_len: int | None = None,
                 sizes=None, unit: int = 64, sorted_first: bool = False) -> Trace:
    """Small random trace for property tests.  `sizes` is an optional alphabet
    of sizes (few values force ties); otherwise sizes are unit * U{1..64}."""
    if num_ops <= 0:
        raise ValueError("num_ops must be positive")
    first = rng.integers(0, num_ops, n)
    if sorted_first:
        first = np.sort(first)
    span = num_ops if max_len is None else max_len
    last = np.minimum(num_ops - 1, first + rng.integers(0, span, n))
    if sizes is None:
        size = unit * rng.integers(1, 65, n)
    else:
        size = np.asarray(sizes, dtype=np.int64)[rng.integers(0, len(sizes), n)]
    return _pack(size, first, last, num_ops)


CONFIG_NAMES = {
    1: "chain256 (256 tensors, 256 ops, seed 1)",
    2: "resnext_batch (1024 traces x 2000 tensors, seeds [2,b])",
    3: "decode100k (100,000 tensors, 4,000 ops, seed 3)",
    4: "ranking1m (1,000,000 tensors, 100,000 ops, seed 4)",
    5: "decode100k plan validation + liveness (seed 5 corruption)",
}
