/*
 * memoplan_oracle.c -- plain, slow, single-threaded CPU oracle of static
 * memory planning (greedy_by_size of Section 2.3, the planner chosen in
 * Section 3.2 of Levental, "Memory Planning for Deep Neural Networks").
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the CPU
 * baseline of the benchmark, never by the product path.  No code is shared
 * with the GPU library.
 *
 * Readings of the thesis fixed here (the text leaves them open):
 *  - a lifetime is the closed op interval [first, last]; two tensors conflict
 *    when they share at least one op;
 *  - a tensor occupies the half-open byte range [offset, offset + size)
 *    (Eq. 2.1: offset_i + mem_i <= offset_j is non-overlap);
 *  - greedy_by_size sorts by size descending, ties by first op ascending, then
 *    by id ascending;
 *  - "fit" for the main policy is the lowest gap that fits (LOWEST_FIT); the
 *    tightest-gap reading of "best fit" is offered as BEST_FIT;
 *  - offsets are never rounded; the peak is max(offset + size) (total_mem of
 *    Eq. 2.1), 0 for an empty trace.
 */
#include "memoplan_oracle.h"

#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Input checks (problem statement of Section 2.3: known sizes and lifetimes) */

/* has_ops == 0 skips the upper bound (plan validation takes no op count). */
static int32_t check_trace(const int64_t* size, const int32_t* first, const int32_t* last,
                           int64_t n, int32_t num_ops, int has_ops) {
    if (n < 0 || num_ops < 0) return MPO_EINVAL;
    if (n > 0 && (!size || !first || !last)) return MPO_EINVAL;
    if (n > INT32_MAX) return MPO_EINVAL;
    int32_t status = MPO_OK;
    uint64_t total = 0; /* saturates at UINT64_MAX */
    for (int64_t i = 0; i < n; ++i) {
        if (size[i] <= 0 || first[i] < 0 || first[i] > last[i] || (has_ops && last[i] >= num_ops))
            status = MPO_EINVAL;
        if (size[i] > 0) {
            uint64_t s = (uint64_t)size[i];
            total = (total > UINT64_MAX - s) ? UINT64_MAX : total + s;
        }
    }
    if (total > (uint64_t)INT64_MAX) status = MPO_EOVERFLOW;
    return status;
}

int32_t mpo_check_trace(const int64_t* size, const int32_t* first, const int32_t* last,
                        int64_t n, int32_t num_ops) {
    return check_trace(size, first, last, n, num_ops, 1);
}

/* ------------------------------------------------------------------------- */
/* Rank order (Section 2.3): size descending, ties by first op ascending,
 * then by id ascending. */

typedef struct {
    int64_t size;
    int32_t first;
    int32_t id;
} rank_key;

static int cmp_rank(const void* pa, const void* pb) {
    const rank_key* a = (const rank_key*)pa;
    const rank_key* b = (const rank_key*)pb;
    if (a->size != b->size) return a->size > b->size ? -1 : 1; /* larger first */
    if (a->first != b->first) return a->first < b->first ? -1 : 1;
    if (a->id != b->id) return a->id < b->id ? -1 : 1;
    return 0;
}

int32_t mpo_rank_order(const int64_t* size, const int32_t* first, int64_t n, int32_t* order_out) {
    if (n < 0 || n > INT32_MAX) return MPO_EINVAL;
    if (n == 0) return MPO_OK;
    if (!size || !first || !order_out) return MPO_EINVAL;
    rank_key* keys = (rank_key*)malloc((size_t)n * sizeof(rank_key));
    if (!keys) return MPO_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        keys[i].size = size[i];
        keys[i].first = first[i];
        keys[i].id = (int32_t)i;
    }
    qsort(keys, (size_t)n, sizeof(rank_key), cmp_rank);
    for (int64_t k = 0; k < n; ++k) order_out[k] = keys[k].id;
    free(keys);
    return MPO_OK;
}

/* ------------------------------------------------------------------------- */
/* Gap search over the byte ranges of the conflicting, already placed tensors.
 * A free gap is a maximal interval of [0, inf) not covered by any range. */

typedef struct {
    int64_t start;
    int64_t end;
} range;

static int cmp_range(const void* pa, const void* pb) {
    const range* a = (const range*)pa;
    const range* b = (const range*)pb;
    if (a->start != b->start) return a->start < b->start ? -1 : 1;
    if (a->end != b->end) return a->end < b->end ? -1 : 1;
    return 0;
}

/* Lowest offset x >= 0 with [x, x + s) disjoint from every range. */
static int64_t lowest_fit(range* r, int64_t k, int64_t s) {
    qsort(r, (size_t)k, sizeof(range), cmp_range);
    int64_t covered_to = 0; /* every byte below covered_to that follows the last gap is taken */
    for (int64_t i = 0; i < k; ++i) {
        if (r[i].start - covered_to >= s) return covered_to;
        if (r[i].end > covered_to) covered_to = r[i].end;
    }
    return covered_to;
}

/* Smallest finite free gap that holds s bytes (lowest start among equals);
 * the unbounded gap above every range only when no finite gap fits. */
static int64_t best_fit(range* r, int64_t k, int64_t s) {
    qsort(r, (size_t)k, sizeof(range), cmp_range);
    int64_t covered_to = 0;
    int64_t best_start = -1, best_len = 0;
    for (int64_t i = 0; i < k; ++i) {
        int64_t gap = r[i].start - covered_to;
        if (gap >= s && (best_start < 0 || gap < best_len)) {
            best_start = covered_to;
            best_len = gap;
        }
        if (r[i].end > covered_to) covered_to = r[i].end;
    }
    return best_start >= 0 ? best_start : covered_to;
}

/* ------------------------------------------------------------------------- */
/* Conflict index: time buckets of width w over the ops; every placed tensor is
 * listed in each bucket its lifetime touches.  Two intersecting lifetimes both
 * contain the op max(first_p, first_t), so a conflicting pair is accepted only
 * in the bucket holding that op, which makes each pair appear exactly once. */

typedef struct {
    int32_t* ids;
    int64_t len;
    int64_t cap;
} id_list;

static int push_id(id_list* l, int32_t id) {
    if (l->len == l->cap) {
        int64_t cap = l->cap ? 2 * l->cap : 16;
        int32_t* p = (int32_t*)realloc(l->ids, (size_t)cap * sizeof(int32_t));
        if (!p) return 0;
        l->ids = p;
        l->cap = cap;
    }
    l->ids[l->len++] = id;
    return 1;
}

/* Places the tensors in the given order: each at the lowest (LOWEST_FIT) or
 * the tightest (BEST_FIT) free gap left by the already placed tensors whose
 * lifetimes intersect its own.  The trace is checked by the caller. */
static int32_t place_in_order(const int64_t* size, const int32_t* first, const int32_t* last,
                              int64_t n, int32_t num_ops, int32_t policy, int32_t bucket_width,
                              const int32_t* order, int64_t* offset_out, int64_t* peak_out) {
    *peak_out = 0;
    if (n == 0) return MPO_OK;
    int64_t nb = ((int64_t)num_ops + bucket_width - 1) / bucket_width;
    id_list* bucket = (id_list*)calloc((size_t)nb, sizeof(id_list));
    range* conf = (range*)malloc((size_t)n * sizeof(range));
    if (!bucket || !conf) {
        free(bucket); free(conf);
        return MPO_EINVAL;
    }
    int32_t status = MPO_OK;
    int64_t peak = 0;
    for (int64_t k = 0; k < n && status == MPO_OK; ++k) {
        int32_t t = order[k];
        int64_t b_lo = first[t] / bucket_width, b_hi = last[t] / bucket_width;
        /* C_t: already placed tensors whose lifetimes intersect t's. */
        int64_t nc = 0;
        for (int64_t b = b_lo; b <= b_hi; ++b) {
            for (int64_t e = 0; e < bucket[b].len; ++e) {
                int32_t p = bucket[b].ids[e];
                if (first[p] > last[t] || first[t] > last[p]) continue;
                int32_t meet = first[p] > first[t] ? first[p] : first[t];
                if (meet / bucket_width != b) continue;
                conf[nc].start = offset_out[p];
                conf[nc].end = offset_out[p] + size[p];
                ++nc;
            }
        }
        int64_t off = (policy == MPO_LOWEST_FIT) ? lowest_fit(conf, nc, size[t])
                                                 : best_fit(conf, nc, size[t]);
        offset_out[t] = off;
        if (off + size[t] > peak) peak = off + size[t];
        for (int64_t b = b_lo; b <= b_hi; ++b)
            if (!push_id(&bucket[b], t)) status = MPO_EINVAL;
    }
    *peak_out = peak;
    for (int64_t b = 0; b < nb; ++b) free(bucket[b].ids);
    free(bucket);
    free(conf);
    return status;
}

int32_t mpo_plan_trace_w(const int64_t* size, const int32_t* first, const int32_t* last,
                         int64_t n, int32_t num_ops, int32_t policy, int32_t bucket_width,
                         int64_t* offset_out, int64_t* peak_out) {
    if (policy != MPO_LOWEST_FIT && policy != MPO_BEST_FIT) return MPO_EINVAL;
    if (bucket_width < 1 || !peak_out) return MPO_EINVAL;
    if (n > 0 && !offset_out) return MPO_EINVAL;
    int32_t st = mpo_check_trace(size, first, last, n, num_ops);
    if (st != MPO_OK) return st;
    *peak_out = 0;
    if (n == 0) return MPO_OK;
    int32_t* order = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    if (!order) return MPO_EINVAL;
    mpo_rank_order(size, first, n, order);
    st = place_in_order(size, first, last, n, num_ops, policy, bucket_width, order, offset_out,
                        peak_out);
    free(order);
    return st;
}

/* About one mean lifetime (only the speed of the conflict index depends on it). */
static int32_t default_bucket_width(const int32_t* first, const int32_t* last, int64_t n,
                                    int32_t num_ops) {
    int64_t w = 1;
    if (n > 0 && first && last) {
        int64_t span = 0;
        for (int64_t i = 0; i < n; ++i)
            if (last[i] >= first[i]) span += (int64_t)last[i] - first[i] + 1;
        w = span / n;
        if (w < 1) w = 1;
        if (w > num_ops && num_ops > 0) w = num_ops;
        if (w > INT32_MAX) w = INT32_MAX;
    }
    return (int32_t)w;
}

int32_t mpo_plan_trace(const int64_t* size, const int32_t* first, const int32_t* last,
                       int64_t n, int32_t num_ops, int32_t policy,
                       int64_t* offset_out, int64_t* peak_out) {
    return mpo_plan_trace_w(size, first, last, n, num_ops, policy,
                            default_bucket_width(first, last, n, num_ops), offset_out, peak_out);
}

/* ------------------------------------------------------------------------- */
/* Live bytes per op: the sum, over tensors alive at op t, of their sizes. */

int32_t mpo_live_bytes_profile(const int64_t* size, const int32_t* first, const int32_t* last,
                               int64_t n, int32_t num_ops, int64_t* live_out,
                               int64_t* max_live_out) {
    if (!max_live_out) return MPO_EINVAL;
    if (num_ops > 0 && !live_out) return MPO_EINVAL;
    int32_t st = mpo_check_trace(size, first, last, n, num_ops);
    if (st != MPO_OK) return st;
    for (int32_t t = 0; t < num_ops; ++t) live_out[t] = 0;
    for (int64_t i = 0; i < n; ++i)
        for (int32_t t = first[i]; t <= last[i]; ++t) live_out[t] += size[i];
    int64_t best = 0;
    for (int32_t t = 0; t < num_ops; ++t)
        if (live_out[t] > best) best = live_out[t];
    *max_live_out = best;
    return MPO_OK;
}

/* ------------------------------------------------------------------------- */
/* Plan validation: the pairwise ordering constraints of Eq. 2.1 say that two
 * tensors with intersecting lifetimes must not overlap in memory. */

int32_t mpo_validate_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                          const int64_t* offset, int64_t n, int64_t* pairs_out,
                          int64_t capacity, int64_t* n_conflicts_out) {
    if (!n_conflicts_out || capacity < 0) return MPO_EINVAL;
    if (capacity > 0 && !pairs_out) return MPO_EINVAL;
    if (n > 0 && !offset) return MPO_EINVAL;
    if (n < 0 || n > INT32_MAX || (n > 0 && (!size || !first || !last))) return MPO_EINVAL;
    /* Each tensor's lifetime and byte range must be well formed; the sum of
     * the sizes plays no part in checking a given plan. */
    for (int64_t i = 0; i < n; ++i)
        if (size[i] <= 0 || first[i] < 0 || first[i] > last[i] || offset[i] < 0 ||
            offset[i] > INT64_MAX - size[i])
            return MPO_EINVAL;
    int64_t count = 0;
    for (int64_t i = 0; i < n; ++i) {
        for (int64_t j = i + 1; j < n; ++j) {
            int lifetimes_meet = first[i] <= last[j] && first[j] <= last[i];
            int bytes_meet = offset[i] < offset[j] + size[j] && offset[j] < offset[i] + size[i];
            if (lifetimes_meet && bytes_meet) {
                if (count < capacity) {
                    pairs_out[2 * count] = i;
                    pairs_out[2 * count + 1] = j;
                }
                ++count;
            }
        }
    }
    *n_conflicts_out = count;
    return count > capacity ? MPO_ENOSPC : MPO_OK;
}

/* ------------------------------------------------------------------------- */
/* Plan application and a write-pattern aliasing probe.  Section 3.3 applies a
 * plan by allocating one slab of total_size bytes and placing every tensor as
 * a view at its offset in it (Listing 5).  The probe replays the ops of the
 * trace in order over such a slab, seen as 32-bit words that are all zero at
 * the start.  At op t:
 *   1. every tensor first used at t writes id + 1 into each word of its byte
 *      range, keeping the larger value where a word already holds one (so
 *      that writers of the same op resolve the same way in any order);
 *   2. every tensor last used at t checks each word of its range: a tensor
 *      that finds any value other than id + 1 is "clobbered";
 *   3. those tensors clear their words to 0.
 * With a valid plan no tensor is clobbered; of every pair that breaks the
 * constraints of Eq. 2.1 at least one tensor is.  Sizes and offsets must be
 * multiples of 4 bytes. */

int32_t mpo_probe_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                       const int64_t* offset, int64_t n, int32_t num_ops,
                       uint8_t* clobbered_out, int64_t* n_clobbered_out) {
    if (!n_clobbered_out || n < 0 || n >= INT32_MAX || num_ops < 0) return MPO_EINVAL;
    if (n > 0 && (!size || !first || !last || !offset || !clobbered_out)) return MPO_EINVAL;
    int64_t words = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (size[i] <= 0 || size[i] % 4 != 0 || offset[i] < 0 || offset[i] % 4 != 0 ||
            offset[i] > INT64_MAX - size[i] || first[i] < 0 || first[i] > last[i] ||
            last[i] >= num_ops)
            return MPO_EINVAL;
        const int64_t end = (offset[i] + size[i]) / 4;
        if (end > words) words = end;
    }
    uint32_t* slab = (uint32_t*)calloc((size_t)(words > 0 ? words : 1), sizeof(uint32_t));
    /* tensors by first op and by last op (counting sort, ids ascending) */
    int64_t* bstart = (int64_t*)calloc((size_t)num_ops + 1, sizeof(int64_t));
    int64_t* dstart = (int64_t*)calloc((size_t)num_ops + 1, sizeof(int64_t));
    int32_t* born = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    int32_t* dies = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    if (!slab || !bstart || !dstart || !born || !dies) {
        free(slab); free(bstart); free(dstart); free(born); free(dies);
        return MPO_EINVAL;
    }
    for (int64_t i = 0; i < n; ++i) {
        ++bstart[first[i] + 1];
        ++dstart[last[i] + 1];
    }
    for (int32_t t = 0; t < num_ops; ++t) {
        bstart[t + 1] += bstart[t];
        dstart[t + 1] += dstart[t];
    }
    for (int64_t i = 0; i < n; ++i) {
        born[bstart[first[i]]++] = (int32_t)i;
        dies[dstart[last[i]]++] = (int32_t)i;
    }
    /* the cursors now hold the ends; the starts are the previous op's ends */
    int64_t count = 0;
    for (int32_t t = 0; t < num_ops; ++t) {
        const int64_t b0 = t ? bstart[t - 1] : 0, b1 = bstart[t];
        const int64_t d0 = t ? dstart[t - 1] : 0, d1 = dstart[t];
        for (int64_t k = b0; k < b1; ++k) {
            const int32_t i = born[k];
            const uint32_t v = (uint32_t)i + 1u;
            for (int64_t w = offset[i] / 4; w < (offset[i] + size[i]) / 4; ++w)
                if (slab[w] < v) slab[w] = v;
        }
        for (int64_t k = d0; k < d1; ++k) {
            const int32_t i = dies[k];
            const uint32_t v = (uint32_t)i + 1u;
            uint8_t bad = 0;
            for (int64_t w = offset[i] / 4; w < (offset[i] + size[i]) / 4; ++w)
                if (slab[w] != v) bad = 1;
            clobbered_out[i] = bad;
            count += bad;
        }
        for (int64_t k = d0; k < d1; ++k) {
            const int32_t i = dies[k];
            for (int64_t w = offset[i] / 4; w < (offset[i] + size[i]) / 4; ++w) slab[w] = 0;
        }
    }
    free(slab); free(bstart); free(dstart); free(born); free(dies);
    *n_clobbered_out = count;
    return MPO_OK;
}

/* ------------------------------------------------------------------------- */
/* bump_allocation: every allocation at the running offset, in the order the
 * allocations happen (first op, then id). */

int32_t mpo_bump_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                      int64_t n, int32_t num_ops, int64_t* offset_out, int64_t* peak_out) {
    if (!peak_out || (n > 0 && !offset_out)) return MPO_EINVAL;
    int32_t st = mpo_check_trace(size, first, last, n, num_ops);
    if (st != MPO_OK) return st;
    /* the order of allocation: a counting sort by first op, ids ascending */
    int64_t* at = (int64_t*)calloc((size_t)num_ops + 1, sizeof(int64_t));
    int64_t* order = (int64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    if (!at || !order) {
        free(at); free(order);
        return MPO_EINVAL;
    }
    for (int64_t i = 0; i < n; ++i) at[first[i] + 1] += 1;
    for (int32_t t = 0; t < num_ops; ++t) at[t + 1] += at[t];
    for (int64_t i = 0; i < n; ++i) order[at[first[i]]++] = i;
    int64_t running = 0;
    for (int64_t k = 0; k < n; ++k) {
        offset_out[order[k]] = running;
        running += size[order[k]];
    }
    *peak_out = running;
    free(at); free(order);
    return MPO_OK;
}

/* ------------------------------------------------------------------------- */
/* The optimum of Eq. 2.1 by exhaustive search over placement orders.  Why the
 * least peak over all orders is the optimum: list the tensors of an optimal
 * plan by offset and place them in that order at the lowest fitting offset;
 * by induction each lands at or below its optimal offset (the ones placed
 * before it sit at or below theirs, which end at or below its own optimal
 * offset whenever their lifetimes meet), so that order reaches the optimum. */

typedef struct {
    const int64_t* size;
    const int32_t* first;
    const int32_t* last;
    int n;
    int64_t off[MPO_OPT_MAX_N];
    int placed[MPO_OPT_MAX_N];  /* placed[i]: tensor i has an offset */
    int64_t best;
    int64_t best_off[MPO_OPT_MAX_N];
} OptSearch;

static int lifetimes_meet(const OptSearch* S, int i, int j) {
    return S->first[i] <= S->last[j] && S->first[j] <= S->last[i];
}

/* Lowest offset for tensor c among the placed tensors: 0 or the end of a
 * placed tensor whose lifetime meets c's, the least such value where c
 * overlaps none of them. */
static int64_t opt_lowest_fit(const OptSearch* S, int c) {
    int64_t best = -1;
    for (int a = -1; a < S->n; ++a) {
        if (a >= 0 && !(S->placed[a] && lifetimes_meet(S, a, c))) continue;
        const int64_t x = a < 0 ? 0 : S->off[a] + S->size[a];
        int free_here = 1;
        for (int j = 0; j < S->n && free_here; ++j)
            if (S->placed[j] && lifetimes_meet(S, j, c) && x < S->off[j] + S->size[j] &&
                S->off[j] < x + S->size[c])
                free_here = 0;
        if (free_here && (best < 0 || x < best)) best = x;
    }
    return best;
}

static void opt_search(OptSearch* S, int depth, int64_t peak) {
    if (depth == S->n) {
        if (peak < S->best) {
            S->best = peak;
            memcpy(S->best_off, S->off, sizeof(S->off));
        }
        return;
    }
    for (int c = 0; c < S->n; ++c) {
        if (S->placed[c]) continue;
        const int64_t x = opt_lowest_fit(S, c);
        S->off[c] = x;
        S->placed[c] = 1;
        opt_search(S, depth + 1, peak > x + S->size[c] ? peak : x + S->size[c]);
        S->placed[c] = 0;
    }
}

int32_t mpo_optimal_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                         int64_t n, int32_t num_ops, int64_t* offset_out, int64_t* peak_out) {
    if (!peak_out || (n > 0 && !offset_out) || n > MPO_OPT_MAX_N) return MPO_EINVAL;
    int32_t st = mpo_check_trace(size, first, last, n, num_ops);
    if (st != MPO_OK) return st;
    OptSearch S;
    memset(&S, 0, sizeof(S));
    S.size = size;
    S.first = first;
    S.last = last;
    S.n = (int)n;
    S.best = INT64_MAX;
    opt_search(&S, 0, 0);
    for (int i = 0; i < S.n; ++i) offset_out[i] = S.best_off[i];
    *peak_out = n > 0 ? S.best : 0;
    return MPO_OK;
}

/* ------------------------------------------------------------------------- */
/* Greedy by Breadth (Section 6, the strategy of Pisarchyk et al.): operators
 * in decreasing breadth -- the sum of the sizes of their input and output
 * tensors -- and, operator by operator, its tensors not yet placed in
 * decreasing size.  In a trace of lifetimes a tensor is an output of its first
 * op and an input of its last op (once when the two coincide). */

typedef struct {
    int64_t key;  /* breadth (sorted descending) or size */
    int32_t idx;  /* op or tensor id (ascending among equal keys) */
} keyed;

static int cmp_keyed(const void* pa, const void* pb) {
    const keyed* a = (const keyed*)pa;
    const keyed* b = (const keyed*)pb;
    if (a->key != b->key) return a->key > b->key ? -1 : 1;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

int32_t mpo_breadth_order(const int64_t* size, const int32_t* first, const int32_t* last,
                          int64_t n, int32_t num_ops, int32_t* order_out) {
    if (n > 0 && !order_out) return MPO_EINVAL;
    int32_t st = mpo_check_trace(size, first, last, n, num_ops);
    if (st != MPO_OK) return st;
    if (n == 0) return MPO_OK;
    int64_t* breadth = (int64_t*)calloc((size_t)num_ops, sizeof(int64_t));
    keyed* ops = (keyed*)malloc((size_t)num_ops * sizeof(keyed));
    keyed* mine = (keyed*)malloc((size_t)n * sizeof(keyed));
    uint8_t* placed = (uint8_t*)calloc((size_t)n, 1);
    /* tensors by op: those first or last used there (a counting sort) */
    int64_t* at = (int64_t*)calloc((size_t)num_ops + 1, sizeof(int64_t));
    int32_t* by_op = (int32_t*)malloc((size_t)(2 * n) * sizeof(int32_t));
    if (!breadth || !ops || !mine || !placed || !at || !by_op) {
        free(breadth); free(ops); free(mine); free(placed); free(at); free(by_op);
        return MPO_EINVAL;
    }
    for (int64_t i = 0; i < n; ++i) {
        breadth[first[i]] += size[i];
        at[first[i] + 1] += 1;
        if (last[i] != first[i]) {
            breadth[last[i]] += size[i];
            at[last[i] + 1] += 1;
        }
    }
    for (int32_t t = 0; t < num_ops; ++t) at[t + 1] += at[t];
    for (int64_t i = 0; i < n; ++i) {
        by_op[at[first[i]]++] = (int32_t)i;
        if (last[i] != first[i]) by_op[at[last[i]]++] = (int32_t)i;
    }
    /* at[t] is now the end of op t's tensors; op t's start is at[t - 1] */
    for (int32_t t = 0; t < num_ops; ++t) {
        ops[t].key = breadth[t];
        ops[t].idx = t;
    }
    qsort(ops, (size_t)num_ops, sizeof(keyed), cmp_keyed);
    int64_t k = 0;
    for (int32_t r = 0; r < num_ops; ++r) {
        const int32_t t = ops[r].idx;
        const int64_t lo = t ? at[t - 1] : 0, hi = at[t];
        int64_t m = 0;
        for (int64_t e = lo; e < hi; ++e) {
            const int32_t i = by_op[e];
            if (placed[i]) continue;
            placed[i] = 1;
            mine[m].key = size[i];
            mine[m].idx = i;
            ++m;
        }
        qsort(mine, (size_t)m, sizeof(keyed), cmp_keyed);
        for (int64_t e = 0; e < m; ++e) order_out[k++] = mine[e].idx;
    }
    free(breadth); free(ops); free(mine); free(placed); free(at); free(by_op);
    return k == n ? MPO_OK : MPO_EINVAL;
}

int32_t mpo_plan_breadth(const int64_t* size, const int32_t* first, const int32_t* last,
                         int64_t n, int32_t num_ops, int32_t policy, int64_t* offset_out,
                         int64_t* peak_out) {
    if (policy != MPO_LOWEST_FIT && policy != MPO_BEST_FIT) return MPO_EINVAL;
    if (!peak_out || (n > 0 && !offset_out)) return MPO_EINVAL;
    int32_t* order = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    if (!order) return MPO_EINVAL;
    int32_t st = mpo_breadth_order(size, first, last, n, num_ops, order);
    if (st == MPO_OK)
        st = place_in_order(size, first, last, n, num_ops, policy,
                            default_bucket_width(first, last, n, num_ops), order, offset_out,
                            peak_out);
    free(order);
    return st;
}

/* ------------------------------------------------------------------------- */
/* Depth of the greedy's dependency structure: the longest chain t1, t2, ...
 * in which each tensor ranks after the previous one and their lifetimes meet
 * (every tensor depends on the earlier-ranked tensors it meets).  Tensors
 * are taken in rank order; a tensor's level is one more than the largest
 * level among the earlier tensors alive at some op of its lifetime, read from
 * a maximum tree over the (compressed) ops that keeps, per op, the largest
 * level of the tensors alive there.  Workload characterisation only. */

typedef struct {
    int32_t* mx;   /* largest level in the node's range */
    int32_t* lazy; /* a level raised over the node's whole range */
    int64_t m;
} max_tree;

static int32_t tree_query(const max_tree* T, int64_t node, int64_t lo, int64_t hi, int64_t a,
                          int64_t b) {
    if (b < lo || hi < a) return 0;
    if (a <= lo && hi <= b) return T->mx[node];
    const int64_t mid = (lo + hi) / 2;
    const int32_t l = tree_query(T, 2 * node, lo, mid, a, b);
    const int32_t r = tree_query(T, 2 * node + 1, mid + 1, hi, a, b);
    int32_t v = l > r ? l : r;
    return v > T->lazy[node] ? v : T->lazy[node];
}

static void tree_raise(max_tree* T, int64_t node, int64_t lo, int64_t hi, int64_t a, int64_t b,
                       int32_t v) {
    if (b < lo || hi < a) return;
    if (a <= lo && hi <= b) {
        if (v > T->mx[node]) T->mx[node] = v;
        if (v > T->lazy[node]) T->lazy[node] = v;
        return;
    }
    const int64_t mid = (lo + hi) / 2;
    tree_raise(T, 2 * node, lo, mid, a, b, v);
    tree_raise(T, 2 * node + 1, mid + 1, hi, a, b, v);
    int32_t w = T->mx[2 * node] > T->mx[2 * node + 1] ? T->mx[2 * node] : T->mx[2 * node + 1];
    if (T->lazy[node] > w) w = T->lazy[node];
    T->mx[node] = w;
}

static int cmp_i32(const void* pa, const void* pb) {
    const int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
    return a < b ? -1 : (a > b ? 1 : 0);
}

static int64_t coord(const int32_t* c, int64_t m, int32_t v) { /* index of v in sorted c */
    int64_t lo = 0, hi = m - 1;
    while (lo < hi) {
        const int64_t mid = (lo + hi) / 2;
        if (c[mid] < v) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

int32_t mpo_dag_depth(const int64_t* size, const int32_t* first, const int32_t* last, int64_t n,
                      int32_t num_ops, int32_t* level_out, int32_t* depth_out) {
    const int32_t st = check_trace(size, first, last, n, num_ops, 0);
    if (st != MPO_OK || !depth_out) return st != MPO_OK ? st : MPO_EINVAL;
    *depth_out = 0;
    if (n == 0) return MPO_OK;
    int32_t* order = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    int32_t* c = (int32_t*)malloc((size_t)(2 * n) * sizeof(int32_t));
    if (!order || !c) {
        free(order);
        free(c);
        return MPO_EINVAL;
    }
    mpo_rank_order(size, first, n, order);
    for (int64_t i = 0; i < n; ++i) {
        c[2 * i] = first[i];
        c[2 * i + 1] = last[i];
    }
    qsort(c, (size_t)(2 * n), sizeof(int32_t), cmp_i32);
    int64_t m = 0;
    for (int64_t i = 0; i < 2 * n; ++i)
        if (m == 0 || c[i] != c[m - 1]) c[m++] = c[i];
    max_tree T = {(int32_t*)calloc((size_t)(4 * m), sizeof(int32_t)),
                  (int32_t*)calloc((size_t)(4 * m), sizeof(int32_t)), m};
    if (!T.mx || !T.lazy) {
        free(order);
        free(c);
        free(T.mx);
        free(T.lazy);
        return MPO_EINVAL;
    }
    int32_t depth = 0;
    for (int64_t k = 0; k < n; ++k) {
        const int32_t t = order[k];
        const int64_t a = coord(c, m, first[t]), b = coord(c, m, last[t]);
        const int32_t lv = tree_query(&T, 1, 0, m - 1, a, b) + 1;
        tree_raise(&T, 1, 0, m - 1, a, b, lv);
        if (level_out) level_out[t] = lv;
        if (lv > depth) depth = lv;
    }
    *depth_out = depth;
    free(order);
    free(c);
    free(T.mx);
    free(T.lazy);
    return MPO_OK;
}

