// Batched greedy-by-size planner: one workgroup per trace, the trace held in LDS.
//
// Method (Section 2.3 greedy_by_size, Section 3.2): tensors are ranked by
// (size desc, first asc, id asc) and each is placed at the lowest offset that
// avoids the byte ranges of the already placed tensors whose lifetimes meet
// its own.  Only lifetime-intersecting pairs interact, so the sequential
// greedy is the same as evaluating each tensor once all of its
// "predecessors" -- intersecting tensors of lower rank -- are placed.  This
// kernel builds the predecessor lists in LDS and lets every lane place its
// tensors as soon as their predecessors are final (a dataflow schedule whose
// length is the depth of the predecessor DAG, not the tensor count).
//
// Positions q: the trace's tensors ordered by (first, id).  For q < q' the
// pair intersects iff first[q'] <= last[q], so tensor q meets exactly the
// positions (q, reach[q]) ahead of it, reach[q] = upper_bound(first, last[q]).
// For such a pair q ranks before q' iff size[q] >= size[q'] (equal sizes are
// ordered by first then id, which is position order) -- the rank comparison
// needs no global sort.
#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr uint32_t kIdleLimit = 1u << 22;  // idle polls without workgroup progress

// Lowest x >= 0 with [x, x+s) clear of every predecessor's [off, off+size).
// Each move jumps past a range that overlaps the candidate window; no offset
// skipped over can fit.  Circular scan: stop after a full lap without moves.
__device__ __forceinline__ uint32_t fit_lowest(const uint16_t* preds, uint32_t pb, uint32_t pe,
                                               const uint32_t* off, const uint32_t* sz,
                                               uint32_t s) {
    const uint32_t k = pe - pb;
    uint32_t x = 0;
    uint32_t c = pb, clean = 0;
    while (clean < k) {
        const uint32_t p = preds[c];
        const uint32_t o = lds_poll(off + p);
        const uint32_t e = o + sz[p];
        if (o < x + s && x < e) {
            x = e;
            clean = 1;
        } else {
            ++clean;
        }
        if (++c == pe) c = pb;
    }
    return x;
}

template <int BLOCK>
__device__ void bitonic_sort_u64(uint64_t* keys, int m) {
    for (int k = 2; k <= m; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < m; i += BLOCK) {
                const int ixj = i ^ j;
                if (ixj > i) {
                    const uint64_t a = keys[i], b = keys[ixj];
                    const bool up = (i & k) == 0;
                    if ((a > b) == up) {
                        keys[i] = b;
                        keys[ixj] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
}

template <int BLOCK, int ITEMS>
__global__ __launch_bounds__(BLOCK) void plan_batch_kernel(
    const int64_t* __restrict__ begin, const int32_t* __restrict__ num_ops,
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, int64_t n_tensors, int32_t cap_n, int32_t cap_pairs,
    int64_t* __restrict__ offset_out, int64_t* __restrict__ peak_out,
    int64_t* __restrict__ lb_out, int32_t* __restrict__ status) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ uint64_t red[BLOCK / kWave];
    __shared__ uint32_t progress_count;

    const size_t N = (size_t)cap_n;
    uint32_t* sz = reinterpret_cast<uint32_t*>(smem);                  // [N] size / unit
    int32_t* fst = reinterpret_cast<int32_t*>(smem + 4 * N);           // [N] first
    uint32_t* off = reinterpret_cast<uint32_t*>(smem + 4 * N);         // [N] offset / unit (reuses fst)
    int32_t* lst = reinterpret_cast<int32_t*>(smem + 8 * N);           // [N] last
    uint32_t* cnt = reinterpret_cast<uint32_t*>(smem + 12 * N);        // [N] pair counts, then cursors
    uint32_t* pbeg = reinterpret_cast<uint32_t*>(smem + 16 * N);       // [N+1] list starts
    uint32_t* diff = reinterpret_cast<uint32_t*>(smem + 20 * N + 4);   // [N+1] live-bytes deltas
    uint16_t* preds = reinterpret_cast<uint16_t*>(smem + 24 * N + 8);  // [cap_pairs]
    uint64_t* keys = reinterpret_cast<uint64_t*>(smem);                // unsorted traces only

    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int64_t lo = begin[b], hi = begin[b + 1];
    const int32_t n_ops = num_ops[b];
    if (lo < 0 || hi < lo || hi > n_tensors || n_ops < 0 || hi - lo > cap_n) {
        if (tid == 0) raise_status(status, MP_EINVAL);
        return;
    }
    const int n = (int)(hi - lo);

    // ---- ingest + checks (ids owned strided: i = tid + k * BLOCK)
    int64_t s_r[ITEMS];
    int32_t f_r[ITEMS], l_r[ITEMS], id_r[ITEMS];
    uint32_t flags = 0;  // bit 0: invalid tensor, bit 1: first not sorted
    uint64_t orv = 0, sum = 0;
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int i = tid + k * BLOCK;
        s_r[k] = 1;
        f_r[k] = 0;
        l_r[k] = 0;
        id_r[k] = i;
        if (i < n) {
            const int64_t s = size[lo + i];
            const int32_t f = first[lo + i], l = last[lo + i];
            s_r[k] = s;
            f_r[k] = f;
            l_r[k] = l;
            if (s <= 0 || f < 0 || f > l || l >= n_ops) flags |= 1u;
            if (s > 0) {
                orv |= (uint64_t)s;
                sum = sat_add(sum, (uint64_t)s);
            }
            fst[i] = f;
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int i = tid + k * BLOCK;
        if (i > 0 && i < n && fst[i] < fst[i - 1]) flags |= 2u;
    }
    flags = block_reduce<BLOCK>(flags, OpOr<uint32_t>(), reinterpret_cast<uint32_t*>(red));
    const uint64_t or_all = block_reduce<BLOCK>(orv, OpOr<uint64_t>(), red);
    const uint64_t total = block_reduce<BLOCK>(sum, OpSatAdd(), red);
    {
        int32_t code = (flags & 1u) ? MP_EINVAL : MP_OK;
        if (total > (uint64_t)INT64_MAX) code = MP_EOVERFLOW;
        if (code != MP_OK) {
            if (tid == 0) raise_status(status, code);
            return;
        }
    }
    if (n == 0) {
        if (tid == 0) {
            peak_out[b] = 0;
            if (lb_out) lb_out[b] = 0;
        }
        return;
    }
    const int sh = __builtin_ctzll(or_all);  // common power-of-two unit of all sizes
    if ((total >> sh) > 0xFFFFFFFEull) {     // offsets are kept as 32-bit unit counts
        if (tid == 0) raise_status(status, MP_ENOSPC);
        return;
    }

    // ---- position order (first, id); recorded traces are normally sorted already
    if (flags & 2u) {
        int m = 1;
        while (m < n) m <<= 1;
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int i = tid + k * BLOCK;
            if (i < m)
                keys[i] = (i < n) ? (((uint64_t)(uint32_t)f_r[k] << 32) | (uint32_t)i) : ~0ull;
        }
        __syncthreads();
        bitonic_sort_u64<BLOCK>(keys, m);
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int q = tid + k * BLOCK;
            if (q < n) id_r[k] = (int32_t)(keys[q] & 0xFFFFFFFFu);
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int q = tid + k * BLOCK;
            if (q < n) {
                s_r[k] = size[lo + id_r[k]];
                f_r[k] = first[lo + id_r[k]];
                l_r[k] = last[lo + id_r[k]];
            }
        }
    }
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        if (q < n) {
            sz[q] = (uint32_t)((uint64_t)s_r[k] >> sh);
            fst[q] = f_r[k];
            lst[q] = l_r[k];
            cnt[q] = 0;
            diff[q] = 0;
        }
    }
    if (tid == 0) {
        diff[n] = 0;
        progress_count = 0;
    }
    __syncthreads();

    // ---- intersecting pairs: count predecessors, live-bytes deltas
    uint32_t su_r[ITEMS];
    int32_t reach_r[ITEMS];
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        su_r[k] = 0;
        reach_r[k] = 0;
        if (q < n) {
            const uint32_t su = sz[q];
            const int32_t l = lst[q];
            int a = q + 1, z = n;  // every position <= q starts no later than l
            while (a < z) {
                const int mid = (a + z) >> 1;
                if (fst[mid] <= l) a = mid + 1;
                else z = mid;
            }
            su_r[k] = su;
            reach_r[k] = a;
            atomicAdd(&diff[q], su);
            atomicAdd(&diff[a], 0u - su);
            uint32_t mine = 0;
            for (int j = q + 1; j < a; ++j) {
                if (su >= sz[j]) atomicAdd(&cnt[j], 1u);
                else ++mine;
            }
            if (mine) atomicAdd(&cnt[q], mine);
        }
    }
    __syncthreads();

    // ---- scans: list starts (exclusive sum of counts) and max live bytes
    uint32_t live_max;
    uint32_t n_pairs;
    {
        const int chunk = (n + BLOCK - 1) / BLOCK;
        const int a0 = min(n, tid * chunk), a1 = min(n, a0 + chunk);
        uint32_t cs = 0, ds = 0;
        for (int i = a0; i < a1; ++i) {
            cs += cnt[i];
            ds += diff[i];
        }
        uint32_t dtot;
        uint32_t cpre = block_exclusive_sum<BLOCK>(cs, &n_pairs, reinterpret_cast<uint32_t*>(red));
        uint32_t dpre = block_exclusive_sum<BLOCK>(ds, &dtot, reinterpret_cast<uint32_t*>(red));
        uint32_t lm = 0;
        for (int i = a0; i < a1; ++i) {
            const uint32_t c = cnt[i];
            pbeg[i] = cpre;
            cpre += c;
            dpre += diff[i];
            lm = lm > dpre ? lm : dpre;
        }
        if (tid == 0) pbeg[n] = n_pairs;
        live_max = block_reduce<BLOCK>(lm, OpMax<uint32_t>(), reinterpret_cast<uint32_t*>(red));
    }
    if (n_pairs > (uint32_t)cap_pairs) {
        if (tid == 0) raise_status(status, MP_ENOSPC);
        return;
    }
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        if (q < n) {
            cnt[q] = pbeg[q];
            off[q] = kUnplaced;
        }
    }
    __syncthreads();

    // ---- predecessor lists
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        if (q < n) {
            const uint32_t su = su_r[k];
            const int a = reach_r[k];
            for (int j = q + 1; j < a; ++j) {
                if (su >= sz[j]) preds[atomicAdd(&cnt[j], 1u)] = (uint16_t)q;
                else preds[atomicAdd(&cnt[q], 1u)] = (uint16_t)j;
            }
        }
    }
    __syncthreads();

    // ---- placement: each tensor as soon as all its predecessors are placed
    {
        uint32_t cur_r[ITEMS];
        uint32_t todo = 0;
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int q = tid + k * BLOCK;
            cur_r[k] = 0;
            if (q < n) {
                todo |= 1u << k;
                cur_r[k] = pbeg[q];
            }
        }
        uint32_t seen = 0, idle = 0;
        bool stuck = false;
        while (todo) {
            bool progress = false;
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                if (todo & (1u << k)) {
                    const int q = tid + k * BLOCK;
                    const uint32_t pe = pbeg[q + 1];
                    uint32_t c = cur_r[k];
                    while (c < pe && lds_poll(off + preds[c]) != kUnplaced) ++c;
                    cur_r[k] = c;
                    if (c == pe) {
                        lds_publish(off + q, fit_lowest(preds, pbeg[q], pe, off, sz, su_r[k]));
                        todo &= ~(1u << k);
                        progress = true;
                    }
                }
            }
            if (progress) {
                atomicAdd(&progress_count, 1u);
            } else {
                const uint32_t now = lds_poll(&progress_count);
                if (now != seen) {
                    seen = now;
                    idle = 0;
                } else if (++idle > kIdleLimit) {
                    stuck = true;  // cannot happen for a valid predecessor DAG
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        if (stuck) raise_status(status, MP_EDEVICE);
    }
    __syncthreads();

    // ---- outputs
    uint32_t pk = 0;
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        if (q < n) {
            const uint32_t o = off[q];
            offset_out[lo + id_r[k]] = (int64_t)((uint64_t)o << sh);
            const uint32_t e = o + su_r[k];
            pk = pk > e ? pk : e;
        }
    }
    pk = block_reduce<BLOCK>(pk, OpMax<uint32_t>(), reinterpret_cast<uint32_t*>(red));
    if (tid == 0) {
        peak_out[b] = (int64_t)((uint64_t)pk << sh);
        if (lb_out) lb_out[b] = (int64_t)((uint64_t)live_max << sh);
    }
}

__global__ void reset_status_kernel(int32_t* status) { *status = MP_OK; }

constexpr int kBatchBlock = 256;

template <int ITEMS>
hipError_t launch_items(const BatchArgs& a, int cap_n, int cap_pairs, size_t lds, hipStream_t st) {
    auto kern = plan_batch_kernel<kBatchBlock, ITEMS>;
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)a.n_traces), dim3(kBatchBlock), lds, st, a.begin,
                       a.num_ops, a.size, a.first, a.last, a.n_tensors, cap_n, cap_pairs,
                       a.offset_out, a.peak_out, a.lb_out, a.status);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_reset_status(int32_t* status, hipStream_t st) {
    hipLaunchKernelGGL(reset_status_kernel, dim3(1), dim3(1), 0, st, status);
    return hipGetLastError();
}

// LDS bytes per workgroup: 24 per tensor slot + 8 + 2 per pair slot.  Traces
// up to 2000 tensors get a budget that lets two workgroups share a CU's
// 160 KiB of LDS.
BatchShape batch_shape(int64_t max_trace_len) {
    BatchShape s{};
    if (max_trace_len < 0 || max_trace_len > MP_BATCH_MAX_TRACE_LEN) return s;
    const int64_t cap_n = max_trace_len < 1 ? 1 : max_trace_len;
    const int64_t fixed = 24 * cap_n + 8;
    const int64_t budget = (fixed <= 48 * 1024) ? 78 * 1024 : 156 * 1024;
    int64_t pairs = (budget - fixed) / 2;
    pairs &= ~(int64_t)7;
    s.cap_n = (int32_t)cap_n;
    s.cap_pairs = (int32_t)pairs;
    s.lds_bytes = (size_t)(fixed + 2 * pairs);
    int items = 1;
    while (items * kBatchBlock < cap_n) items <<= 1;
    s.items = items;
    s.ok = true;
    return s;
}

hipError_t launch_plan_batch(const BatchArgs& a, hipStream_t st) {
    const BatchShape s = batch_shape(a.max_trace_len);
    if (!s.ok) return hipErrorInvalidValue;
    switch (s.items) {
        case 1: return launch_items<1>(a, s.cap_n, s.cap_pairs, s.lds_bytes, st);
        case 2: return launch_items<2>(a, s.cap_n, s.cap_pairs, s.lds_bytes, st);
        case 4: return launch_items<4>(a, s.cap_n, s.cap_pairs, s.lds_bytes, st);
        case 8: return launch_items<8>(a, s.cap_n, s.cap_pairs, s.lds_bytes, st);
        case 16: return launch_items<16>(a, s.cap_n, s.cap_pairs, s.lds_bytes, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mp
