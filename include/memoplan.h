/*
 * memoplan.h -- C ABI of the MI355X (gfx950) static memory planner.
 *
 * What it computes (Levental, "Memory Planning for Deep Neural Networks"):
 * given the byte size and the lifetime [first, last] (closed interval of op
 * indices) of every intermediate tensor of a recorded trace, assign each
 * tensor a byte offset in one arena so that no two tensors whose lifetimes
 * intersect overlap in memory (the offline dynamic-storage-allocation problem
 * of Section 2.3; the non-overlap constraint is the ordering constraint of
 * Eq. 2.1).  Offsets come from greedy_by_size (Section 2.3, the default
 * planner of Section 3.2): tensors are taken by size descending, ties by first
 * op ascending, then by id ascending; each is put at the lowest offset at
 * which it does not overlap any already placed tensor whose lifetime meets
 * its own.  The arena size (total_mem of Eq. 2.1, the slab of Section 3.3)
 * is max(offset + size), 0 for an empty trace.
 *
 * Conventions shared by every entry point
 *  - All array arguments are DEVICE pointers owned by the caller; the library
 *    never allocates device memory, never frees, never synchronises.  Work is
 *    enqueued on `stream` (a hipStream_t passed as void*; NULL = null stream).
 *  - Tensor id = array index (in a batch: index within its trace).  Sizes are
 *    int64 bytes, lifetimes int32 op indices, offsets int64 bytes.
 *  - Return value (host, synchronous): MP_OK when the work was enqueued;
 *    MP_EINVAL for bad host arguments (NULL pointer where data is needed,
 *    negative counts, counts above 2^40, unknown policy, workspace too
 *    small), in which case nothing is launched; MP_EDEVICE when a launch
 *    fails.
 *  - Data-dependent errors are found on the device and folded into the
 *    caller's device int32 `*status_out` with an atomic minimum, so the word
 *    is sticky: it holds the most negative code of every call since the last
 *    mp_status_reset on it.  Codes: MP_EINVAL for size <= 0, first < 0,
 *    first > last or last >= num_ops; MP_EOVERFLOW when the sizes of a trace
 *    sum past INT64_MAX; MP_ENOSPC when a documented capacity is exceeded;
 *    MP_EDEVICE for an internal failure of a kernel.  Outputs of a call are
 *    unspecified when it raised a code.
 *  - Calls that share a status word or outputs on different streams race.
 */
#ifndef MEMOPLAN_H
#define MEMOPLAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MP_OK 0
#define MP_EINVAL (-1)
#define MP_ENOSPC (-2)
#define MP_EOVERFLOW (-3)
#define MP_EDEVICE (-4)

/* Fit policy.  LOWEST_FIT: lowest gap that fits.  BEST_FIT: tightest finite
 * gap that fits (lowest start among equals), the space above every conflicting
 * tensor only when no finite gap fits -- a reading of the best-fit rule of
 * Section 2.3. */
#define MP_LOWEST_FIT 0
#define MP_BEST_FIT 1

/* Longest trace (tensors) the batched planner accepts. */
#define MP_BATCH_MAX_TRACE_LEN 4096

/* Human-readable name of a status code (static storage). */
const char* mp_status_string(int32_t status);

/* Enqueue *status_out = MP_OK on `stream` (one single-thread kernel).
 * Returns MP_EINVAL for a NULL pointer, MP_EDEVICE if the launch fails. */
int32_t mp_status_reset(int32_t* status_out, void* stream);

/* Greedy-by-size plans for many independent traces in one launch (one
 * workgroup per trace).
 *   begin[n_traces + 1] int64: trace b owns tensors [begin[b], begin[b+1]) of
 *                        the concatenated arrays; 0 <= begin[b] <= begin[b+1]
 *                        <= n_tensors (checked on device, MP_EINVAL).
 *   num_ops[n_traces]  int32: op count of each trace (lifetimes < num_ops[b]).
 *   size, first, last  [n_tensors] (int64, int32, int32).
 *   n_tensors          length of the concatenated arrays (bounds check of begin).
 *   max_trace_len      host bound on begin[b+1] - begin[b], 0..4096: sizes the
 *                      per-workgroup LDS without reading begin on the host; a
 *                      longer trace sets MP_EINVAL (plan it with mp_plan_trace).
 *   policy             MP_LOWEST_FIT or MP_BEST_FIT.
 *   offset_out[n_tensors] int64, peak_out[n_traces] int64 (arena bytes),
 *   lb_out[n_traces]   int64 or NULL: max over ops of the live bytes, a lower
 *                      bound on any valid arena size.
 *   workspace          device memory of mp_workspace_bytes(MP_OP_PLAN_BATCH,
 *                      n_tensors, 0, n_traces) bytes; contents need no
 *                      initialisation; not used after the call completes.
 * Every valid trace is planned.  A trace is held in LDS (its intersecting
 * pairs as one-byte list entries) when its sizes sum to less than 2^31 units
 * of 2^ctz(OR of sizes), its pairs fit mp_batch_pair_capacity(max_trace_len)
 * and at most 32 of its tensors meet a tensor born more than 223 positions
 * later (and, under BEST_FIT, no tensor meets more than 256 others);
 * otherwise the same workgroup plans it on a general path (64-bit offsets,
 * working lists in the workspace, O(n^2) work per trace), with the same
 * results. */
int32_t mp_plan_batch(const int64_t* begin, int64_t n_traces, const int32_t* num_ops,
                      const int64_t* size, const int32_t* first, const int32_t* last,
                      int64_t n_tensors, int64_t max_trace_len, int32_t policy,
                      int64_t* offset_out, int64_t* peak_out, int64_t* lb_out,
                      void* workspace, size_t workspace_bytes, int32_t* status_out,
                      void* stream);

/* Intersecting pairs per trace that mp_plan_batch holds in LDS for a given
 * max_trace_len (host query, no device work); a trace with more takes the
 * general path.  -1 when max_trace_len is out of range. */
int64_t mp_batch_pair_capacity(int64_t max_trace_len);

/* Greedy-by-size plan of one trace of any length, using the whole device
 * (a persistent kernel: workgroups take tensors in rank order, in blocks of
 * 32 consecutive ranks per XCD, and each fits its tensor once the
 * earlier-ranked tensors that meet it are placed).
 *   size, first, last [n] (int64, int32, int32), 0 <= n < 2^30.
 *   offset_out[n] int64, peak_out: one device int64 (arena bytes).
 *   policy: MP_LOWEST_FIT or MP_BEST_FIT.
 *   workspace: mp_workspace_bytes(MP_OP_PLAN_TRACE, n, num_ops, 1) bytes on
 *              the current device (it depends on the CU count); its contents
 *              need no initialisation.
 * Every valid trace is planned: offsets are kept as 32-bit counts of
 * 2^ctz(OR of sizes) while the sizes sum to less than 2^32 - 1 such units,
 * as 64-bit counts beyond (chosen on the device); a tensor with more
 * earlier-ranked intersecting tensors than its workgroup's buffer holds
 * (131072, or 32768 with 64-bit counts) waits until all of them are placed,
 * takes one of two shared buffers of n ranges and is fitted there.
 * Tensors need not be sorted by first.
 * Test build: compiled with MP_DEBUG_WAIT (libmemoplan_dbgwait.so), this
 * call reads the environment variable MEMOPLAN_DEBUG_WAIT on each call; "wide"
 * makes every wait for late predecessors take its widest form, "tight"
 * besides caps the late list at 8, so tensors with more wait during their
 * collection and the call reports MP_EDEVICE.  Offsets are exact either way;
 * both only exercise paths the schedule rarely reaches. */
int32_t mp_plan_trace(const int64_t* size, const int32_t* first, const int32_t* last, int64_t n,
                      int32_t num_ops, int32_t policy, int64_t* offset_out, int64_t* peak_out,
                      void* workspace, size_t workspace_bytes, int32_t* status_out,
                      void* stream);

/* Workspace bytes of the call selected by `op` (host query, no device
 * work), from the number of tensors, the largest op count and the number of
 * traces: MP_OP_PLAN_BATCH (n_tensors, n_traces), MP_OP_PLAN_TRACE
 * (n_tensors), MP_OP_LIVE_BYTES (max_num_ops), MP_OP_VALIDATE (n_tensors; a
 * pairs_out capacity of at most n_tensors), MP_OP_VALIDATE_BATCH (n_tensors,
 * n_traces; capacity at most n_tensors), MP_OP_PROBE (n_tensors,
 * max_num_ops; the default capacity), MP_OP_BUMP (n_tensors).  The
 * single-trace planner's size depends on the current device (its CU count).
 * Returns 0 for an unknown op or out-of-range sizes (negative, or counts above
 * 2^40). */
#define MP_OP_LIVE_BYTES 1
#define MP_OP_VALIDATE 2
#define MP_OP_PLAN_TRACE 3
#define MP_OP_VALIDATE_BATCH 4
#define MP_OP_PLAN_BATCH 5
#define MP_OP_PROBE 6
#define MP_OP_BUMP 7
size_t mp_workspace_bytes(int32_t op, int64_t n_tensors, int64_t max_num_ops, int64_t n_traces);

/* The same sizes with the output capacity explicit: MP_OP_LIVE_BYTES (uses
 * num_ops), MP_OP_VALIDATE (uses n_tensors and capacity, the pairs_out
 * capacity), MP_OP_PLAN_TRACE (uses n_tensors), MP_OP_VALIDATE_BATCH (uses
 * n_tensors, capacity and the number of traces passed as num_ops),
 * MP_OP_PLAN_BATCH (n_tensors and the number of traces passed as num_ops),
 * MP_OP_PROBE (uses n_tensors, num_ops and capacity, the number of lane
 * events to hold; 0 asks for 16 n_tensors + 65536), MP_OP_BUMP (uses
 * n_tensors).  Returns 0 for an unknown op or out-of-range sizes. */
size_t mp_workspace_size(int32_t op, int64_t n_tensors, int64_t num_ops, int64_t capacity);

/* Per-op live bytes of one trace (the quantity whose maximum lower-bounds
 * total_mem of Eq. 2.1: every tensor alive at an op needs its own bytes).
 *   live_out[num_ops] int64: live_out[t] = sum of size[i] over first[i] <= t <= last[i].
 *   max_live_out: one device int64, max over t (0 when num_ops == 0).
 *   workspace: mp_workspace_size(MP_OP_LIVE_BYTES, n, num_ops, 0) bytes. */
int32_t mp_live_bytes_profile(const int64_t* size, const int32_t* first, const int32_t* last,
                              int64_t n, int32_t num_ops, int64_t* live_out,
                              int64_t* max_live_out, void* workspace, size_t workspace_bytes,
                              int32_t* status_out, void* stream);

/* mp_live_bytes_profile for callers that cannot allocate device memory
 * (code under stream capture, tight serving loops, harnesses that forbid
 * hipMalloc): same arguments and results, no workspace.  Its scratch (a
 * counter and the prefix sum's tile partials, about 64 KiB) is a static
 * device array that each GPU the library runs on holds until the process
 * ends, looked up once per device on the first call there.  num_ops above
 * MP_LIVE_NOALLOC_MAX_OPS is MP_EINVAL from the call (use
 * mp_live_bytes_profile).  Nothing is allocated, freed or synchronised.
 * Every call on one GPU shares that scratch: calls that overlap in time on
 * the same GPU (different streams, or different host threads) race and must
 * be ordered by the caller.  MP_EDEVICE if the scratch cannot be resolved. */
#define MP_LIVE_NOALLOC_MAX_OPS (1 << 24)
int32_t mp_live_bytes_profile_noalloc(const int64_t* size, const int32_t* first,
                                      const int32_t* last, int64_t n, int32_t num_ops,
                                      int64_t* live_out, int64_t* max_live_out,
                                      int32_t* status_out, void* stream);

/* Plan validation against the pairwise constraints of Eq. 2.1: every pair
 * i < j whose lifetimes intersect and whose byte ranges [offset, offset +
 * size) overlap.
 *   pairs_out[2 * capacity] int64: (i, j) pairs in lexicographic order; only
 *                      the first `capacity` are written.
 *   n_conflicts_out:   one device int64, always the exact number of pairs;
 *                      MP_ENOSPC on the status word when it exceeds capacity.
 *   hints:             0 or MP_HINT_SORTED_FIRST (below).
 *   workspace:         mp_workspace_size(MP_OP_VALIDATE, n, 0, capacity) bytes.
 * Data errors (MP_EINVAL): size <= 0, first < 0, first > last, offset < 0,
 * offset + size > INT64_MAX.  Tensors need not be sorted by first. */
int32_t mp_validate_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                         const int64_t* offset, int64_t n, int64_t* pairs_out, int64_t capacity,
                         int64_t* n_conflicts_out, int32_t hints, void* workspace,
                         size_t workspace_bytes, int32_t* status_out, void* stream);

/* hints for the validation calls: MP_HINT_SORTED_FIRST promises that first
 * is non-decreasing within every trace (recorded traces are, since tensors
 * are numbered in allocation order).  The sorting kernels are then not
 * enqueued; a broken promise is reported as MP_EINVAL. */
#define MP_HINT_SORTED_FIRST 1

/* mp_validate_plan over a batch of independent traces (trace b = tensors
 * [begin[b], begin[b+1]) with begin[0] == 0 and begin[n_traces] == n_tensors,
 * checked on device).  Pairs use indices into the concatenated arrays; no
 * pair crosses traces.
 *   max_trace_len:  0, or a bound on the tensors of every trace, at most
 *                   MP_BATCH_MAX_TRACE_LEN.  With MP_HINT_SORTED_FIRST a
 *                   nonzero bound selects the path that holds each trace in
 *                   one workgroup's LDS (count per trace, scan, write); a
 *                   trace above the bound is then MP_EINVAL on device.
 *                   Otherwise the bound is not used.
 *   workspace:      mp_workspace_size(MP_OP_VALIDATE_BATCH, n_tensors,
 *                   n_traces, capacity) bytes; contents need no
 *                   initialisation. */
int32_t mp_validate_batch(const int64_t* begin, int64_t n_traces, const int64_t* size,
                          const int32_t* first, const int32_t* last, const int64_t* offset,
                          int64_t n_tensors, int64_t max_trace_len, int64_t* pairs_out,
                          int64_t capacity, int64_t* n_conflicts_out, int32_t hints,
                          void* workspace, size_t workspace_bytes, int32_t* status_out,
                          void* stream);

/* A plan applied and exercised: the slab of Section 3.3 (one allocation of
 * total_size bytes, every tensor a view at its offset, as in Listing 5),
 * probed by replaying the ops in order over its 32-bit words, zeroed first.
 * At op t every tensor first used at t writes id + 1 into each word of its
 * range, keeping the larger value where a word already holds one; then every
 * tensor last used at t checks its words -- a tensor that finds another value
 * is clobbered -- and clears them to 0.  A valid plan clobbers nothing; of
 * every pair breaking Eq. 2.1 at least one tensor is clobbered (the result
 * does not depend on the order of the writers of one op).
 *   size, first, last, offset [n] (int64, int32, int32, int64): sizes and
 *              offsets multiples of 4 bytes, 0 <= first <= last < num_ops.
 *   slab:      device memory of slab_bytes >= max(offset + size) bytes (the
 *              plan's peak), 4-byte aligned; overwritten.
 *   clobbered_out[n] uint8: 1 for a clobbered tensor, else 0.
 *   n_clobbered_out: one device int64, the number of clobbered tensors.
 *   workspace: mp_workspace_size(MP_OP_PROBE, n, num_ops, capacity) bytes,
 *              or more; contents need no initialisation.  `capacity` is the
 *              number of (tensor, 256-byte slab tile) pairs the tiled replay
 *              holds, 0 for 16 n + 65536; the call takes the largest capacity
 *              that workspace_bytes holds.
 * The replay is split by address: one wave per tile of 64 words replays, in
 * op order, the events of the tensors covering the tile.  A plan with more
 * pairs than the capacity is replayed op by op by one workgroup instead
 * (same results, far slower).
 * Data errors (MP_EINVAL on the status word): a size <= 0, a size or offset
 * not a multiple of 4, a negative offset, an invalid lifetime, a slab smaller
 * than the plan.  A workspace too small even for the op-by-op replay is
 * MP_EINVAL from the call. */
int32_t mp_probe_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                      const int64_t* offset, int64_t n, int32_t num_ops, void* slab,
                      size_t slab_bytes, uint8_t* clobbered_out, int64_t* n_clobbered_out,
                      void* workspace, size_t workspace_bytes, int32_t* status_out, void* stream);

/* bump_allocation, the baseline strategy of Section 2.3: allocations are
 * taken in the order they happen -- by first op, ties by id -- and each goes
 * at a running offset that then grows by its size; nothing is reused, so the
 * peak is the sum of the sizes.
 *   begin[n_traces + 1] int64: trace bounds (0 = begin[0] <= ... <=
 *              begin[n_traces] = n), or NULL for one trace of n tensors.
 *   size, first, last [n]: as for mp_plan_trace; every last < num_ops (for a
 *              batch, num_ops bounds every trace's op count).
 *   offset_out[n] int64, peak_out[n_traces] int64 (one value when begin is
 *              NULL): the offsets and each trace's sum of sizes.
 *   workspace: mp_workspace_size(MP_OP_BUMP, n, 0, 0) bytes, contents need no
 *              initialisation.
 * Data errors (on the status word): MP_EINVAL for a size <= 0, a lifetime
 * outside [0, num_ops) or inverted, or bad trace bounds; MP_EOVERFLOW when
 * the sizes of all traces together exceed INT64_MAX. */
int32_t mp_bump_plan(const int64_t* begin, int64_t n_traces, const int64_t* size,
                     const int32_t* first, const int32_t* last, int64_t n, int32_t num_ops,
                     int64_t* offset_out, int64_t* peak_out, void* workspace,
                     size_t workspace_bytes, int32_t* status_out, void* stream);

/* The optimum of Eq. 2.1 (the least total_mem under its pairwise
 * constraints; the thesis's mip strategy) for tiny traces, by exhaustive
 * search: the least peak over all placement orders with each tensor at the
 * lowest offset that overlaps no placed tensor whose lifetime meets its own
 * (an optimal plan listed by offset is such an order).  One workgroup per
 * trace; subtrees whose partial peak reaches the best found are cut, and a
 * trace stops once the best equals its live-bytes lower bound.
 *   begin[n_traces + 1] int64, num_ops[n_traces] int32, size/first/last
 *              [n_tensors]: as for mp_plan_batch; each trace at most
 *              MP_OPT_MAX_N tensors.
 *   offset_out[n_tensors]: one optimal plan (optimal plans are not unique);
 *   peak_out[n_traces]: the optimum.
 * Data errors (MP_EINVAL on the status word): a trace over MP_OPT_MAX_N
 * tensors or with bad bounds, an invalid tensor; MP_EOVERFLOW when a trace's
 * sizes exceed INT64_MAX.  Time grows like n! in the worst case. */
#define MP_OPT_MAX_N 12
int32_t mp_optimal_batch(const int64_t* begin, int64_t n_traces, const int32_t* num_ops,
                         const int64_t* size, const int32_t* first, const int32_t* last,
                         int64_t n_tensors, int64_t* offset_out, int64_t* peak_out,
                         int32_t* status_out, void* stream);

/* Greedy by Breadth, the strategy of Pisarchyk et al. that Section 6
 * describes: operators in decreasing breadth (the sum of the sizes of their
 * input and output tensors; lower op first on ties), and for each operator its
 * tensors not yet placed in decreasing size (lower id first), each at the
 * lowest (MP_LOWEST_FIT) or tightest (MP_BEST_FIT) gap left by the placed
 * tensors whose lifetimes meet its own -- the same fit rules as greedy by
 * size.  A tensor is an output of its first op and an input of its last op
 * (once when they coincide): the trace records no other operator membership.
 *   begin, num_ops, size, first, last, n_tensors: as for mp_plan_batch; each
 *              trace at most MP_BREADTH_MAX_TRACE_LEN tensors.
 *   offset_out[n_tensors], peak_out[n_traces]: offsets and peaks.
 * One workgroup per trace, the trace held in LDS; no workspace.
 * Data errors (on the status word): MP_EINVAL for an invalid tensor, bad trace
 * bounds or a trace over MP_BREADTH_MAX_TRACE_LEN tensors; MP_EOVERFLOW when
 * a trace's sizes exceed INT64_MAX. */
#define MP_BREADTH_MAX_TRACE_LEN 2048
int32_t mp_plan_breadth_batch(const int64_t* begin, int64_t n_traces, const int32_t* num_ops,
                              const int64_t* size, const int32_t* first, const int32_t* last,
                              int64_t n_tensors, int32_t policy, int64_t* offset_out,
                              int64_t* peak_out, int32_t* status_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif
