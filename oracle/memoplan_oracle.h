/*
 * memoplan_oracle.h -- plain, single-threaded CPU oracle of static memory
 * planning by greedy-by-size (Levental, "Memory Planning for Deep Neural
 * Networks", Section 2.3 and Section 3.2).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or
 * call this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code with the GPU library.
 *
 * All pointers are host pointers owned by the caller.  All arithmetic is
 * integer.  Status codes (same values as the product ABI, defined separately):
 *   0 ok, -1 invalid argument or trace, -2 output capacity too small,
 *   -3 sum of sizes exceeds INT64_MAX.
 * When several data errors are present the most negative code is returned.
 */
#ifndef MEMOPLAN_ORACLE_H
#define MEMOPLAN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MPO_OK 0
#define MPO_EINVAL (-1)
#define MPO_ENOSPC (-2)
#define MPO_EOVERFLOW (-3)

#define MPO_LOWEST_FIT 0
#define MPO_BEST_FIT 1

/* Trace check: every size > 0 and 0 <= first <= last < num_ops (lifetimes are
 * closed op intervals), and the sizes sum to at most INT64_MAX. */
int32_t mpo_check_trace(const int64_t* size, const int32_t* first, const int32_t* last,
                        int64_t n, int32_t num_ops);

/* Greedy-by-size placement order: ids sorted by (size descending, first
 * ascending, id ascending).  order_out[k] = id placed k-th. */
int32_t mpo_rank_order(const int64_t* size, const int32_t* first, int64_t n, int32_t* order_out);

/* Greedy-by-size offsets (Section 2.3, greedy_by_size; Section 3.2).  Tensors
 * are taken in rank order; each is put at the lowest (LOWEST_FIT) or the
 * tightest (BEST_FIT) free gap left by the already placed tensors whose
 * lifetimes intersect its own.  *peak_out = max(offset + size), 0 if n == 0
 * (total_mem of Eq. 2.1, the slab size of Section 3.3). */
int32_t mpo_plan_trace(const int64_t* size, const int32_t* first, const int32_t* last,
                       int64_t n, int32_t num_ops, int32_t policy,
                       int64_t* offset_out, int64_t* peak_out);

/* Same as mpo_plan_trace with an explicit time-bucket width of the conflict
 * index (any width >= 1 gives the same result; exposed for tests). */
int32_t mpo_plan_trace_w(const int64_t* size, const int32_t* first, const int32_t* last,
                         int64_t n, int32_t num_ops, int32_t policy, int32_t bucket_width,
                         int64_t* offset_out, int64_t* peak_out);

/* live_out[t] = sum of sizes of tensors with first <= t <= last, t in
 * [0, num_ops); *max_live_out = max_t live_out[t] (0 if num_ops == 0). */
int32_t mpo_live_bytes_profile(const int64_t* size, const int32_t* first, const int32_t* last,
                               int64_t n, int32_t num_ops, int64_t* live_out,
                               int64_t* max_live_out);

/* Every pair i < j whose lifetimes intersect and whose byte ranges
 * [offset, offset + size) overlap (the pairwise constraints of Eq. 2.1).
 * Input errors (-1): size <= 0, first < 0, first > last, offset < 0,
 * offset + size > INT64_MAX; the sum of the sizes is not checked here.
 * pairs_out[2k], pairs_out[2k+1] = (i, j) in lexicographic order; at most
 * `capacity` pairs are written; *n_conflicts_out is always the exact count and
 * the status is -2 when it exceeds capacity. */
int32_t mpo_validate_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                          const int64_t* offset, int64_t n, int64_t* pairs_out,
                          int64_t capacity, int64_t* n_conflicts_out);

/* Write-pattern aliasing probe of a plan (plan application of Section 3.3,
 * Listing 5): the ops are replayed in order over a zeroed slab of 32-bit
 * words; at op t the tensors first used at t write id + 1 into their words
 * (keeping the larger value), then the tensors last used at t check that
 * their words hold id + 1 (clobbered_out[i] = 1 otherwise) and clear them.
 * Sizes and offsets must be multiples of 4.  *n_clobbered_out = the count. */
int32_t mpo_probe_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                       const int64_t* offset, int64_t n, int32_t num_ops,
                       uint8_t* clobbered_out, int64_t* n_clobbered_out);

/* bump_allocation (Section 2.3, the baseline strategy): allocations are taken
 * in the order they happen -- by first op, ties by id -- and each goes at a
 * running offset that then grows by its size; no memory is reused.
 * *peak_out = the sum of the sizes. */
int32_t mpo_bump_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                      int64_t n, int32_t num_ops, int64_t* offset_out, int64_t* peak_out);

/* The optimum of Eq. 2.1 for tiny traces (n <= MPO_OPT_MAX_N, else -1): the
 * least peak over all n! placement orders, each tensor placed at the lowest
 * offset where it overlaps no earlier-placed tensor whose lifetime meets its
 * own.  offset_out gets the plan of the first optimal order in lexicographic
 * order of the ids. */
#define MPO_OPT_MAX_N 12
int32_t mpo_optimal_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                         int64_t n, int32_t num_ops, int64_t* offset_out, int64_t* peak_out);

/* Greedy by Breadth (the strategy of Pisarchyk et al. that Section 6
 * describes): operators in decreasing breadth, the sum of the sizes of their
 * input and output tensors (ties: lower op first), and for each operator its
 * tensors not yet placed in decreasing size (ties: lower id first).  Reading
 * for a trace of lifetimes: a tensor is an output of its first op and an
 * input of its last op, counted once when the two coincide.
 * mpo_breadth_order writes the order; mpo_plan_breadth places the tensors in
 * it with the fit policy of mpo_plan_trace. */
int32_t mpo_breadth_order(const int64_t* size, const int32_t* first, const int32_t* last,
                          int64_t n, int32_t num_ops, int32_t* order_out);
int32_t mpo_plan_breadth(const int64_t* size, const int32_t* first, const int32_t* last,
                         int64_t n, int32_t num_ops, int32_t policy, int64_t* offset_out,
                         int64_t* peak_out);

/* Depth of greedy_by_size's dependency structure (workload characterisation,
 * not a planning result): level[t] = 1 + the largest level among the
 * earlier-ranked tensors whose lifetimes meet t's (1 when there are none);
 * *depth_out = the largest level, 0 for n == 0.  level_out may be NULL. */
int32_t mpo_dag_depth(const int64_t* size, const int32_t* first, const int32_t* last, int64_t n,
                      int32_t num_ops, int32_t* level_out, int32_t* depth_out);

#ifdef __cplusplus
}
#endif

#endif
