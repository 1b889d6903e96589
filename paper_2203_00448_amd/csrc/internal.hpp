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
};

struct BatchShape {
    bool ok;
    int32_t cap_n;      // tensor slots per workgroup
    int32_t cap_pairs;  // predecessor-list slots per workgroup
    int32_t items;      // tensor slots per thread
    size_t lds_bytes;   // dynamic LDS per workgroup
};

BatchShape batch_shape(int64_t max_trace_len);
hipError_t launch_reset_status(int32_t* status, hipStream_t st);
hipError_t launch_plan_batch(const BatchArgs& a, hipStream_t st);

}  // namespace mp
