"""Independent, definitional Python versions used to pin the oracle.

These are deliberately different computations from the oracle's C code:
no sorting of conflicts, no time buckets, no sweeps.  They follow the
definitions directly (Section 2.3: offline DSA, greedy_by_size; Eq. 2.1) and
are only usable on small traces.
"""
from __future__ import annotations

import itertools

import numpy as np


def conflict(f, l, i, j) -> bool:
    """Closed op intervals [f, l] share at least one op."""
    return i != j and f[i] <= l[j] and f[j] <= l[i]


def disjoint_bytes(oi, si, oj, sj) -> bool:
    """Half-open byte ranges do not overlap (Eq. 2.1 ordering constraint)."""
    return oi + si <= oj or oj + sj <= oi


def rank_order(size, first):
    return sorted(range(len(size)), key=lambda i: (-int(size[i]), int(first[i]), i))


def _feasible(x, s, placed):
    return all(disjoint_bytes(x, s, o, z) for o, z in placed)


def lowest_fit_candidates(s, placed):
    """Lowest feasible x using the candidate set {0} U {ends}, checked O(K^2)."""
    cands = [0] + [o + z for o, z in placed]
    return min(x for x in cands if _feasible(x, s, placed))


def best_fit_candidates(s, placed):
    """Tightest free gap holding s (lowest start among equals); the unbounded
    gap above all ranges only if no finite gap fits.  Gaps are enumerated from
    their starts: a start is 0 or an end, not covered by any range."""
    starts = sorted({0} | {o + z for o, z in placed})
    best = None
    for g in starts:
        if any(o <= g < o + z for o, z in placed):
            continue
        above = [o for o, z in placed if o >= g]
        if not above:
            continue  # the unbounded gap
        length = min(above) - g
        if length >= s and (best is None or (length, g) < best):
            best = (length, g)
    if best is not None:
        return best[1]
    return max([o + z for o, z in placed], default=0)


def greedy_definitional(size, first, last, policy: int = 0):
    """Greedy-by-size straight from the definition: earlier-ranked tensors
    whose lifetimes meet t's are found by an all-pairs loop."""
    n = len(size)
    order = rank_order(size, first)
    off = [None] * n
    for k, t in enumerate(order):
        placed = [(off[p], int(size[p])) for p in order[:k] if conflict(first, last, p, t)]
        s = int(size[t])
        off[t] = lowest_fit_candidates(s, placed) if policy == 0 else best_fit_candidates(s, placed)
    peak = max((off[i] + int(size[i]) for i in range(n)), default=0)
    return off, peak


def place_in_order(order, size, first, last, stack: bool):
    """Place tensors in the given order; lowest fitting gap (stack=False) or on
    top of every conflicting placed tensor (stack=True).  Returns the peak."""
    off = {}
    for t in order:
        placed = [(off[p], int(size[p])) for p in off if conflict(first, last, p, t)]
        s = int(size[t])
        if stack:
            off[t] = max((o + z for o, z in placed), default=0)
        else:
            off[t] = lowest_fit_candidates(s, placed)
    return max((off[i] + int(size[i]) for i in off), default=0)


def brute_force_opt(size, first, last, stack: bool) -> int:
    """Optimum of Eq. 2.1 for tiny traces: the best peak over all placement
    orders (either placement rule reaches the optimum: sort an optimal plan
    by offset and place in that order)."""
    n = len(size)
    return min(place_in_order(p, size, first, last, stack)
               for p in itertools.permutations(range(n)))


def live_profile_bruteforce(size, first, last, num_ops):
    live = np.zeros(num_ops, dtype=np.int64)
    for t in range(num_ops):
        live[t] = sum(int(size[i]) for i in range(len(size)) if first[i] <= t <= last[i])
    return live


def intersecting_pairs_band(first, last):
    """All i < j with intersecting lifetimes, by sorting on the first op and
    walking forward while the other tensor starts no later than this one ends."""
    n = len(first)
    order = sorted(range(n), key=lambda i: (int(first[i]), i))
    pairs = set()
    for a, i in enumerate(order):
        for j in order[a + 1:]:
            if first[j] > last[i]:
                break
            pairs.add((min(i, j), max(i, j)))
    return pairs


def breadth_order_definitional(size, first, last):
    """Greedy by Breadth order written out: each op's breadth is the bytes of
    the tensors it produces (first op) or last reads (last op), once for a
    tensor that does both; ops by breadth descending then index; within an op
    its tensors not yet taken by size descending then id."""
    n = len(size)
    ops = {}
    for i in range(n):
        for t in {int(first[i]), int(last[i])}:
            ops.setdefault(t, []).append(i)
    breadth = {t: sum(int(size[i]) for i in ids) for t, ids in ops.items()}
    taken, order = set(), []
    for t in sorted(ops, key=lambda t: (-breadth[t], t)):
        mine = sorted((i for i in ops[t] if i not in taken), key=lambda i: (-int(size[i]), i))
        taken.update(mine)
        order += mine
    return order


def place_in_given_order(order, size, first, last, policy):
    off = [None] * len(size)
    for k, t in enumerate(order):
        placed = [(off[p], int(size[p])) for p in order[:k] if conflict(first, last, p, t)]
        s = int(size[t])
        off[t] = lowest_fit_candidates(s, placed) if policy == 0 else best_fit_candidates(s, placed)
    return off, max((off[i] + int(size[i]) for i in range(len(size))), default=0)


def interleaved_trace(k):
    """(size, first, last, num_ops, offsets, peak) of a trace with a closed-form
    lowest-fit plan: 2k tensors of 64 B alive at op 0, the odd ids also at op
    1, then one of 64 B alive at op 1 only.  In rank order (equal sizes: id
    order) the first 2k pack at 64 j; the last meets only the odd ones, whose
    ranges are k disjoint intervals, and goes at 0.  Peak 128 k."""
    n = 2 * k + 1
    first = np.zeros(n, np.int32)
    first[-1] = 1
    last = np.zeros(n, np.int32)
    last[1:2 * k:2] = 1
    last[-1] = 1
    off = np.append(64 * np.arange(2 * k, dtype=np.int64), 0)
    return np.full(n, 64, np.int64), first, last, 2, off, 128 * k


def packed_wide_trace(n):
    """Closed-form lowest-fit plan of n - 1 tensors of 4 KiB (ids 1..n-1) and
    one of 64 B (id 0), all alive at ops 0-1: the large ones rank first and
    pack in id order, the small one goes on top at 4096 (n - 1)."""
    size = np.full(n, 4096, np.int64)
    size[0] = 64
    off = np.append(4096 * (n - 1), 4096 * np.arange(n - 1, dtype=np.int64))
    return size, np.zeros(n, np.int32), np.ones(n, np.int32), 2, off, 4096 * (n - 1) + 64
