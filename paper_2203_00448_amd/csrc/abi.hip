// C ABI entry points: host-side argument checks, then launches on the
// caller's stream.  No allocation, no synchronisation.
#include "internal.hpp"

using namespace mp;

namespace {

int32_t launched(hipError_t e) { return e == hipSuccess ? MP_OK : MP_EDEVICE; }

// Largest element count (tensors, ops, traces, pair capacity) any size
// computation takes: far beyond any device, small enough that byte counts
// of a few dozen bytes per element stay within 64 bits.
constexpr int64_t kMaxElems = (int64_t)1 << 40;

}  // namespace

extern "C" const char* mp_status_string(int32_t status) {
    switch (status) {
        case MP_OK: return "ok";
        case MP_EINVAL: return "invalid argument or trace";
        case MP_ENOSPC: return "capacity exceeded";
        case MP_EOVERFLOW: return "sum of sizes exceeds INT64_MAX";
        case MP_EDEVICE: return "device launch or execution failure";
        default: return "unknown status";
    }
}

extern "C" int32_t mp_status_reset(int32_t* status_out, void* stream) {
    if (!status_out) return MP_EINVAL;
    return launched(launch_reset_status(status_out, static_cast<hipStream_t>(stream)));
}

extern "C" int64_t mp_batch_pair_capacity(int64_t max_trace_len) {
    const BatchShape s = batch_shape(max_trace_len);
    return s.ok ? (int64_t)s.cap_pairs : -1;
}

extern "C" int32_t mp_plan_batch(const int64_t* begin, int64_t n_traces, const int32_t* num_ops,
                                 const int64_t* size, const int32_t* first, const int32_t* last,
                                 int64_t n_tensors, int64_t max_trace_len, int32_t policy,
                                 int64_t* offset_out, int64_t* peak_out, int64_t* lb_out,
                                 void* workspace, size_t workspace_bytes, int32_t* status_out,
                                 void* stream) {
    if (n_traces < 0 || n_traces > INT32_MAX || n_tensors < 0 || n_tensors > kMaxElems ||
        !status_out)
        return MP_EINVAL;
    if (policy != MP_LOWEST_FIT && policy != MP_BEST_FIT) return MP_EINVAL;
    if (!batch_shape(max_trace_len).ok) return MP_EINVAL;
    if (!begin) return MP_EINVAL;
    if (n_traces > 0 && (!num_ops || !peak_out || !workspace)) return MP_EINVAL;
    if (n_tensors > 0 && (!size || !first || !last || !offset_out)) return MP_EINVAL;
    if (workspace_bytes < plan_batch_workspace_bytes(n_tensors, n_traces)) return MP_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (n_traces == 0) return MP_OK;
    BatchArgs a{begin,      n_traces,      num_ops,    size,     first,  last,       n_tensors,
                max_trace_len, offset_out, peak_out, lb_out, status_out, workspace, policy};
    return launched(launch_plan_batch(a, st));
}

extern "C" size_t mp_workspace_size(int32_t op, int64_t n_tensors, int64_t num_ops,
                                    int64_t capacity) {
    if (n_tensors < 0 || num_ops < 0 || capacity < 0) return 0;
    if (n_tensors > kMaxElems || num_ops > kMaxElems || capacity > kMaxElems) return 0;
    switch (op) {
        case MP_OP_LIVE_BYTES:
            return num_ops > INT32_MAX ? 0 : live_workspace_bytes((int32_t)num_ops);
        case MP_OP_VALIDATE:
            return validate_workspace_bytes(n_tensors, capacity, 1);
        case MP_OP_PLAN_BATCH:
            return num_ops > INT32_MAX ? 0 : plan_batch_workspace_bytes(n_tensors, num_ops);
        case MP_OP_VALIDATE_BATCH:
            return num_ops > INT32_MAX ? 0 : validate_workspace_bytes(n_tensors, capacity, num_ops);
        case MP_OP_PLAN_TRACE:
            return n_tensors >= (int64_t)1 << 30 ? 0 : plan_trace_workspace_bytes(n_tensors);
        case MP_OP_BUMP:
            return bump_workspace_bytes(n_tensors);
        case MP_OP_PROBE:
            return num_ops > INT32_MAX ? 0
                                       : probe_workspace_bytes(n_tensors, (int32_t)num_ops,
                                                               capacity);
        default:
            return 0;
    }
}

extern "C" size_t mp_workspace_bytes(int32_t op, int64_t n_tensors, int64_t max_num_ops,
                                     int64_t n_traces) {
    if (n_tensors < 0 || n_tensors > kMaxElems || max_num_ops < 0 || max_num_ops > INT32_MAX ||
        n_traces < 0 || n_traces > INT32_MAX)
        return 0;
    switch (op) {
        case MP_OP_LIVE_BYTES:
            return live_workspace_bytes((int32_t)max_num_ops);
        case MP_OP_VALIDATE:
            return validate_workspace_bytes(n_tensors, n_tensors, 1);
        case MP_OP_VALIDATE_BATCH:
            return validate_workspace_bytes(n_tensors, n_tensors, n_traces > 0 ? n_traces : 1);
        case MP_OP_PLAN_TRACE:
            return n_tensors >= (int64_t)1 << 30 ? 0 : plan_trace_workspace_bytes(n_tensors);
        case MP_OP_PLAN_BATCH:
            return plan_batch_workspace_bytes(n_tensors, n_traces);
        case MP_OP_BUMP:
            return bump_workspace_bytes(n_tensors);
        case MP_OP_PROBE:
            return probe_workspace_bytes(n_tensors, (int32_t)max_num_ops, 0);
        default:
            return 0;
    }
}

extern "C" int32_t mp_live_bytes_profile(const int64_t* size, const int32_t* first,
                                         const int32_t* last, int64_t n, int32_t num_ops,
                                         int64_t* live_out, int64_t* max_live_out, void* workspace,
                                         size_t workspace_bytes, int32_t* status_out,
                                         void* stream) {
    if (n < 0 || num_ops < 0 || !status_out || !max_live_out || !workspace) return MP_EINVAL;
    if (n > 0 && (!size || !first || !last)) return MP_EINVAL;
    if (num_ops > 0 && !live_out) return MP_EINVAL;
    if (workspace_bytes < live_workspace_bytes(num_ops)) return MP_EINVAL;
    return launched(launch_live_profile(size, first, last, n, num_ops, live_out, max_live_out,
                                        workspace, status_out, static_cast<hipStream_t>(stream)));
}

extern "C" int32_t mp_live_bytes_profile_noalloc(const int64_t* size, const int32_t* first,
                                                 const int32_t* last, int64_t n, int32_t num_ops,
                                                 int64_t* live_out, int64_t* max_live_out,
                                                 int32_t* status_out, void* stream) {
    if (n < 0 || num_ops < 0 || num_ops > MP_LIVE_NOALLOC_MAX_OPS || !status_out || !max_live_out)
        return MP_EINVAL;
    if (n > 0 && (!size || !first || !last)) return MP_EINVAL;
    if (num_ops > 0 && !live_out) return MP_EINVAL;
    return launched(launch_live_profile_noalloc(size, first, last, n, num_ops, live_out,
                                                max_live_out, status_out,
                                                static_cast<hipStream_t>(stream)));
}

namespace {

int32_t validate_common(const int64_t* begin, int64_t n_seg, const int64_t* size,
                        const int32_t* first, const int32_t* last, const int64_t* offset,
                        int64_t n, int64_t max_seg, int64_t* pairs_out, int64_t capacity,
                        int64_t* n_conflicts_out, int32_t hints, void* workspace,
                        size_t workspace_bytes, int32_t* status_out, void* stream) {
    if (n < 0 || n > INT32_MAX - 1 || capacity < 0 || capacity > kMaxElems || !status_out ||
        !n_conflicts_out || !workspace)
        return MP_EINVAL;
    if (n > 0 && (!size || !first || !last || !offset)) return MP_EINVAL;
    if (capacity > 0 && !pairs_out) return MP_EINVAL;
    if (hints & ~MP_HINT_SORTED_FIRST) return MP_EINVAL;
    if (max_seg < 0 || max_seg > MP_BATCH_MAX_TRACE_LEN) return MP_EINVAL;
    if (workspace_bytes < validate_workspace_bytes(n, capacity, begin ? n_seg : 1))
        return MP_EINVAL;
    return launched(launch_validate(begin, n_seg, size, first, last, offset, n, max_seg,
                                    pairs_out, capacity, n_conflicts_out,
                                    (hints & MP_HINT_SORTED_FIRST) != 0, workspace, status_out,
                                    static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" int32_t mp_validate_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                                    const int64_t* offset, int64_t n, int64_t* pairs_out,
                                    int64_t capacity, int64_t* n_conflicts_out, int32_t hints,
                                    void* workspace, size_t workspace_bytes, int32_t* status_out,
                                    void* stream) {
    return validate_common(nullptr, 1, size, first, last, offset, n, 0, pairs_out, capacity,
                           n_conflicts_out, hints, workspace, workspace_bytes, status_out, stream);
}

extern "C" int32_t mp_validate_batch(const int64_t* begin, int64_t n_traces, const int64_t* size,
                                     const int32_t* first, const int32_t* last,
                                     const int64_t* offset, int64_t n_tensors,
                                     int64_t max_trace_len, int64_t* pairs_out, int64_t capacity,
                                     int64_t* n_conflicts_out, int32_t hints, void* workspace,
                                     size_t workspace_bytes, int32_t* status_out, void* stream) {
    if (!begin || n_traces < 1 || n_traces > INT32_MAX) return MP_EINVAL;
    return validate_common(begin, n_traces, size, first, last, offset, n_tensors, max_trace_len,
                           pairs_out, capacity, n_conflicts_out, hints, workspace,
                           workspace_bytes, status_out, stream);
}

extern "C" int32_t mp_plan_trace(const int64_t* size, const int32_t* first, const int32_t* last,
                                 int64_t n, int32_t num_ops, int32_t policy, int64_t* offset_out,
                                 int64_t* peak_out, void* workspace, size_t workspace_bytes,
                                 int32_t* status_out, void* stream) {
    if (n < 0 || n >= (int64_t)1 << 30 || num_ops < 0 || !status_out || !peak_out || !workspace)
        return MP_EINVAL;
    if (policy != MP_LOWEST_FIT && policy != MP_BEST_FIT) return MP_EINVAL;
    if (n > 0 && (!size || !first || !last || !offset_out)) return MP_EINVAL;
    if (workspace_bytes < plan_trace_workspace_bytes(n)) return MP_EINVAL;
    return launched(launch_plan_trace(size, first, last, n, num_ops, policy, offset_out, peak_out,
                                      workspace, status_out, static_cast<hipStream_t>(stream)));
}

extern "C" int32_t mp_probe_plan(const int64_t* size, const int32_t* first, const int32_t* last,
                                 const int64_t* offset, int64_t n, int32_t num_ops, void* slab,
                                 size_t slab_bytes, uint8_t* clobbered_out,
                                 int64_t* n_clobbered_out, void* workspace,
                                 size_t workspace_bytes, int32_t* status_out, void* stream) {
    if (n < 0 || n >= INT32_MAX || num_ops < 0 || !status_out || !n_clobbered_out || !workspace)
        return MP_EINVAL;
    if (n > 0 && (!size || !first || !last || !offset || !clobbered_out || !slab))
        return MP_EINVAL;
    if (slab && (reinterpret_cast<uintptr_t>(slab) & 3)) return MP_EINVAL;
    if (probe_capacity(n, num_ops, workspace_bytes) < 0) return MP_EINVAL;
    return launched(launch_probe(size, first, last, offset, n, num_ops, slab, slab ? slab_bytes : 0,
                                 clobbered_out, n_clobbered_out, workspace, workspace_bytes,
                                 status_out, static_cast<hipStream_t>(stream)));
}

extern "C" int32_t mp_bump_plan(const int64_t* begin, int64_t n_traces, const int64_t* size,
                                const int32_t* first, const int32_t* last, int64_t n,
                                int32_t num_ops, int64_t* offset_out, int64_t* peak_out,
                                void* workspace, size_t workspace_bytes, int32_t* status_out,
                                void* stream) {
    if (n < 0 || n >= INT32_MAX || num_ops < 0 || !status_out || !peak_out || !workspace)
        return MP_EINVAL;
    if (begin && (n_traces < 0 || n_traces >= INT32_MAX)) return MP_EINVAL;
    if (n > 0 && (!size || !first || !last || !offset_out)) return MP_EINVAL;
    if (workspace_bytes < bump_workspace_bytes(n)) return MP_EINVAL;
    return launched(launch_bump(begin, begin ? n_traces : 1, size, first, last, n, num_ops,
                                offset_out, peak_out, workspace, status_out,
                                static_cast<hipStream_t>(stream)));
}

extern "C" int32_t mp_optimal_batch(const int64_t* begin, int64_t n_traces,
                                    const int32_t* num_ops, const int64_t* size,
                                    const int32_t* first, const int32_t* last,
                                    int64_t n_tensors, int64_t* offset_out, int64_t* peak_out,
                                    int32_t* status_out, void* stream) {
    if (n_traces < 0 || n_traces > INT32_MAX || n_tensors < 0 || !status_out) return MP_EINVAL;
    if (n_traces > 0 && (!begin || !num_ops || !peak_out)) return MP_EINVAL;
    if (n_tensors > 0 && (!size || !first || !last || !offset_out)) return MP_EINVAL;
    return launched(launch_optimal(begin, n_traces, num_ops, size, first, last, n_tensors,
                                   offset_out, peak_out, status_out,
                                   static_cast<hipStream_t>(stream)));
}

extern "C" int32_t mp_plan_breadth_batch(const int64_t* begin, int64_t n_traces,
                                         const int32_t* num_ops, const int64_t* size,
                                         const int32_t* first, const int32_t* last,
                                         int64_t n_tensors, int32_t policy, int64_t* offset_out,
                                         int64_t* peak_out, int32_t* status_out, void* stream) {
    if (n_traces < 0 || n_traces > INT32_MAX || n_tensors < 0 || !status_out) return MP_EINVAL;
    if (policy != MP_LOWEST_FIT && policy != MP_BEST_FIT) return MP_EINVAL;
    if (n_traces > 0 && (!begin || !num_ops || !peak_out)) return MP_EINVAL;
    if (n_tensors > 0 && (!size || !first || !last || !offset_out)) return MP_EINVAL;
    return launched(launch_breadth(begin, n_traces, num_ops, size, first, last, n_tensors, policy,
                                   offset_out, peak_out, status_out,
                                   static_cast<hipStream_t>(stream)));
}
