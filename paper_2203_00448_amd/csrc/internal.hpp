// Internal launch interface between the C ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "memoplan.h"

namespace mp {

struct BatchArgs {
    const int64_t* begin;
    int64_t n_traces;
    const int32_t* num_ops;
    const int64_t* size;
    const int32_t* first;
    const int32_t* last;
    int64_t n_tensors;
    int64_t max_trace_len;
    int64_t* offset_out;
    int64_t* peak_out;
    int64_t* lb_out;
    int32_t* status;
    void* workspace;  // plan_batch_workspace_bytes(n_tensors, n_traces)
    int32_t policy;   // MP_LOWEST_FIT or MP_BEST_FIT
};

struct BatchShape {
    bool ok;
    int32_t cap_n;      // tensor slots per workgroup
    int32_t cap_pairs;  // left-list entries (one byte each) per trace in LDS
    int32_t items;      // tensor slots per thread
    int32_t block;      // threads per workgroup (one trace each)
    size_t lds_bytes;   // dynamic LDS per workgroup
};

BatchShape batch_shape(int64_t max_trace_len);
size_t plan_batch_workspace_bytes(int64_t n_tensors, int64_t n_traces);
hipError_t launch_reset_status(int32_t* status, hipStream_t st);
hipError_t launch_plan_batch(const BatchArgs& a, hipStream_t st);

// write-pattern aliasing probe of a plan (probe.hip)
size_t probe_workspace_bytes(int64_t n, int32_t num_ops, int64_t capacity);
int64_t probe_capacity(int64_t n, int32_t num_ops, size_t workspace_bytes);
hipError_t launch_probe(const int64_t* size, const int32_t* first, const int32_t* last,
                        const int64_t* offset, int64_t n, int32_t num_ops, void* slab,
                        size_t slab_bytes, uint8_t* clob, int64_t* n_clob, void* ws,
                        size_t ws_bytes, int32_t* status, hipStream_t st);

}  // namespace mp

namespace mp {

// bump_allocation and the exact optimum (strategies.hip)
size_t bump_workspace_bytes(int64_t n);
hipError_t launch_bump(const int64_t* begin, int64_t n_seg, const int64_t* size,
                       const int32_t* first, const int32_t* last, int64_t n, int32_t num_ops,
                       int64_t* offset_out, int64_t* peak_out, void* ws, int32_t* status,
                       hipStream_t st);
hipError_t launch_optimal(const int64_t* begin, int64_t n_traces, const int32_t* num_ops,
                          const int64_t* size, const int32_t* first, const int32_t* last,
                          int64_t n_tensors, int64_t* offset_out, int64_t* peak_out,
                          int32_t* status, hipStream_t st);

// Greedy by Breadth (breadth.hip)
hipError_t launch_breadth(const int64_t* begin, int64_t n_traces, const int32_t* num_ops,
                          const int64_t* size, const int32_t* first, const int32_t* last,
                          int64_t n_tensors, int32_t policy, int64_t* offset_out,
                          int64_t* peak_out, int32_t* status, hipStream_t st);

// device-wide prefix sums (scan.hip)
size_t scan_workspace_bytes(int64_t n);
hipError_t device_scan_i64(int64_t* data, int64_t n, bool inclusive, int64_t* partial,
                           unsigned long long* max_out, hipStream_t st,
                           const uint32_t* skip = nullptr);

// stable LSD radix sort of (u64 key, u32 value) pairs (radix.hip)
size_t radix_workspace_bytes(int64_t n);
hipError_t radix_sort_pairs(uint64_t* k0, uint32_t* v0, uint64_t* k1, uint32_t* v1, int64_t n,
                            int begin_bit, int end_bit, void* ws, bool* in_alt, hipStream_t st,
                            const uint32_t* skip = nullptr, const int64_t* n_live = nullptr);

// liveness profile (live.hip)
size_t live_workspace_bytes(int32_t num_ops);
hipError_t launch_live_profile(const int64_t* size, const int32_t* first, const int32_t* last,
                               int64_t n, int32_t num_ops, int64_t* live_out, int64_t* max_out,
                               void* ws, int32_t* status, hipStream_t st);
size_t live_noalloc_scratch_bytes();
hipError_t launch_live_profile_noalloc(const int64_t* size, const int32_t* first,
                                       const int32_t* last, int64_t n, int32_t num_ops,
                                       int64_t* live_out, int64_t* max_out, int32_t* status,
                                       hipStream_t st);


// plan validation (validate.hip); begin == nullptr means one trace of n tensors
size_t validate_workspace_bytes(int64_t n, int64_t capacity, int64_t n_seg);
hipError_t launch_validate(const int64_t* begin, int64_t n_seg, const int64_t* size,
                           const int32_t* first, const int32_t* last, const int64_t* off,
                           int64_t n, int64_t max_seg, int64_t* pairs, int64_t cap,
                           int64_t* n_out, bool assume_sorted, void* ws, int32_t* status,
                           hipStream_t st);


// single-trace planner (plan_trace.hip)
size_t plan_trace_workspace_bytes(int64_t n);
hipError_t launch_plan_trace(const int64_t* size, const int32_t* first, const int32_t* last,
                             int64_t n, int32_t num_ops, int32_t policy, int64_t* offset_out,
                             int64_t* peak_out, void* ws, int32_t* status, hipStream_t st);

}  // namespace mp
