// Greedy by Breadth, the strategy of Pisarchyk et al. that Section 6 sets
// beside greedy_by_size: operators in decreasing breadth (the bytes of their
// input and output tensors, lower op first on ties), and for each operator
// its tensors not yet placed in decreasing size (lower id first).  In a trace
// of lifetimes a tensor is an output of its first op and an input of its last
// op, once when the two coincide.  Each tensor then goes at the lowest (or the
// tightest) gap left by the placed tensors whose lifetimes meet its own.
//
// One workgroup per trace, the trace in LDS.  A tensor is placed with the op
// that comes first in the op order among its two ops, so the whole order is a
// sort of the tensors by (breadth of that op desc, op, size desc, id): op
// breadths from a histogram over ops, then a bitonic sort of the indices.
// Placement is one tensor after another, two barriers a step: all waves find
// the placed tensors whose lifetimes meet the tensor and compact them into
// LDS (a ballot prefix within a wave, one LDS atomic per wave); then wave 0
// tests every candidate start (0 or one of their ends) on its lanes and a
// shuffle minimum picks the answer -- or, for the lowest fit with at most 64
// neighbours, a walk from 0 past the overlapping neighbours.
#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr int kBBlock = 512;
constexpr int kBMax = MP_BREADTH_MAX_TRACE_LEN;

struct BreadthShared {
    int64_t size[kBMax];
    int64_t off[kBMax];  // -1 until placed
    int32_t first[kBMax];
    int32_t last[kBMax];
    uint16_t order[kBMax];
    union {  // the ranking's keys, then (while placing) the neighbour list
        struct {
            int64_t bkey[kBMax];  // breadth of the op the tensor is placed with
            int32_t op[kBMax];
        };
        uint16_t nb[kBMax];  // placed tensors meeting the current one
    };
    uint32_t n_nb;
    int32_t bad;
};
// two workgroups per CU (160 KB of LDS)
static_assert(sizeof(BreadthShared) <= 80 * 1024 - 128, "LDS of the breadth planner");

__device__ __forceinline__ int64_t readlane64(int64_t v, int q) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, q);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), q);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Lexicographic (a0, a1) minimum over the wave; every lane gets it.
__device__ __forceinline__ void wave_min2(uint64_t& a0, uint64_t& a1) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const uint64_t b0 = __shfl_xor(a0, o, kWave), b1 = __shfl_xor(a1, o, kWave);
        if (b0 < a0 || (b0 == a0 && b1 < a1)) {
            a0 = b0;
            a1 = b1;
        }
    }
}

__global__ __launch_bounds__(kBBlock) void breadth_kernel(
    const int64_t* __restrict__ begin, const int32_t* __restrict__ num_ops,
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, int64_t n_tensors, int32_t policy,
    int64_t* __restrict__ offset_out, int64_t* __restrict__ peak_out,
    int32_t* __restrict__ status) {
    __shared__ BreadthShared S;
    __shared__ uint64_t red[kBBlock / kWave];
    const int tid = threadIdx.x;
    const int64_t b0 = begin[blockIdx.x], b1 = begin[blockIdx.x + 1];
    if (b0 < 0 || b1 > n_tensors || b1 < b0 || b1 - b0 > kBMax) {
        if (tid == 0) raise_status(status, MP_EINVAL);
        return;
    }
    const int n = (int)(b1 - b0);
    const int32_t T = num_ops[blockIdx.x];
    if (tid == 0) S.bad = 0;
    __syncthreads();
    uint64_t acc = 0;
    for (int i = tid; i < n; i += kBBlock) {
        const int64_t s = size[b0 + i];
        const int32_t f = first[b0 + i], l = last[b0 + i];
        if (s <= 0 || f < 0 || f > l || l >= T) atomicOr(&S.bad, 1);
        else acc = sat_add(acc, (uint64_t)s);
        S.size[i] = s;
        S.first[i] = f;
        S.last[i] = l;
        S.off[i] = -1;
    }
    acc = block_reduce<kBBlock>(acc, OpSatAdd(), red);
    if (S.bad) {
        if (tid == 0) raise_status(status, MP_EINVAL);
        return;
    }
    if (acc > (uint64_t)INT64_MAX) {
        if (tid == 0) raise_status(status, MP_EOVERFLOW);
        return;
    }
    // each tensor's two op breadths, and the op it is placed with: a
    // histogram over ops (a tensor adds its size at its first op and, if
    // different, at its last), held in the LDS of the offsets while it is
    // needed; more ops than that: a count over all pairs
    if (T <= kBMax) {
        int64_t* hist = S.off;
        for (int o = tid; o < T; o += kBBlock) hist[o] = 0;
        __syncthreads();
        for (int i = tid; i < n; i += kBBlock) {
            const int32_t f = S.first[i], l = S.last[i];
            const unsigned long long s = (unsigned long long)S.size[i];
            atomicAdd(reinterpret_cast<unsigned long long*>(&hist[f]), s);
            if (l != f) atomicAdd(reinterpret_cast<unsigned long long*>(&hist[l]), s);
        }
        __syncthreads();
        for (int i = tid; i < n; i += kBBlock) {
            const int32_t f = S.first[i], l = S.last[i];
            const int64_t bf = hist[f], bl = hist[l];
            S.bkey[i] = bf >= bl ? bf : bl;
            S.op[i] = bf >= bl ? f : l;
        }
        __syncthreads();
        for (int i = tid; i < n; i += kBBlock) S.off[i] = -1;
    } else {
        for (int i = tid; i < n; i += kBBlock) {
            const int32_t f = S.first[i], l = S.last[i];
            int64_t bf = 0, bl = 0;
            for (int j = 0; j < n; ++j) {
                const int32_t fj = S.first[j], lj = S.last[j];
                const int64_t sj = S.size[j];
                bf += (fj == f || lj == f) ? sj : 0;
                bl += (fj == l || lj == l) ? sj : 0;
            }
            S.bkey[i] = bf >= bl ? bf : bl;
            S.op[i] = bf >= bl ? f : l;
        }
    }
    __syncthreads();
    // rank order (breadth desc, op asc, size desc, id asc): a bitonic sort of
    // the indices, padded to a power of two with indices >= n that go last
    int np2 = 1;
    while (np2 < n) np2 <<= 1;
    for (int i = tid; i < np2; i += kBBlock) S.order[i] = (uint16_t)i;
    __syncthreads();
    auto ranks_before = [&](int a, int b) {
        if (b >= n) return a < n || a < b;
        if (a >= n) return false;
        const int64_t ba = S.bkey[a], bb = S.bkey[b];
        if (ba != bb) return ba > bb;
        const int32_t oa = S.op[a], ob = S.op[b];
        if (oa != ob) return oa < ob;
        const int64_t sa = S.size[a], sb = S.size[b];
        if (sa != sb) return sa > sb;
        return a < b;
    };
    for (int k = 2; k <= np2; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < (np2 >> 1); i += kBBlock) {
                const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1)), hi = lo | j;
                const int a = S.order[lo], b = S.order[hi];
                const bool up = (lo & k) == 0;
                if (up ? ranks_before(b, a) : ranks_before(a, b)) {
                    S.order[lo] = (uint16_t)b;
                    S.order[hi] = (uint16_t)a;
                }
            }
            __syncthreads();
        }
    }
    const int lane = tid & (kWave - 1);
    const uint64_t below = (1ull << lane) - 1ull;  // lanes before this one
    if (tid == 0) S.n_nb = 0;
    __syncthreads();
    int64_t peak = 0;
    for (int k = 0; k < n; ++k) {
        const int t = S.order[k];
        const int32_t ft = S.first[t], lt = S.last[t];
        const int64_t st = S.size[t];
        // placed tensors meeting t, compacted into S.nb (any order)
        for (int j0 = tid - lane; j0 < n; j0 += kBBlock) {
            const int j = j0 + lane;
            const bool hit = j < n && S.off[j] >= 0 && S.first[j] <= lt && ft <= S.last[j];
            const uint64_t b = __ballot(hit);
            if (b) {
                uint32_t base = 0;
                if (lane == 0) base = atomicAdd(&S.n_nb, (uint32_t)__popcll(b));
                base = (uint32_t)__shfl(base, 0, kWave);
                if (hit) S.nb[base + __popcll(b & below)] = (uint16_t)j;
            }
        }
        __syncthreads();
        if (tid < kWave && policy != MP_BEST_FIT && (int)S.n_nb <= kWave) {
            // wave 0, lowest fit with at most 64 neighbours (one a lane): from
            // 0, jump to the highest end among the neighbours overlapping
            // [x, x + st) until none does; each jump skips only blocked starts
            const int m = (int)S.n_nb;
            int64_t oq = 0, eq = INT64_MIN;  // no neighbour: never overlaps
            if (lane < m) {
                const int j = S.nb[lane];
                oq = S.off[j];
                eq = oq + S.size[j];
            }
            int64_t x = 0;
            while (true) {
                uint64_t ov = __ballot(oq < x + st && x < eq);
                if (!ov) break;
                int64_t v = x;
                for (; ov; ov &= ov - 1) v = max(v, readlane64(eq, (int)__builtin_ctzll(ov)));
                x = v;
            }
            if (lane == 0) {
                S.off[t] = x;
                S.n_nb = 0;
            }
            peak = max(peak, x + st);
        } else if (tid < kWave) {  // wave 0: candidate starts, 0 (c == m) and each neighbour's end
            const int m = (int)S.n_nb;
            uint64_t key0 = ~0ull, key1 = ~0ull;  // lowest: (x, 0); best: (gap, x)
            for (int c0 = 0; c0 <= m; c0 += kWave) {
                const int c = c0 + lane;
                int64_t x = 0;
                if (c < m) {
                    const int j = S.nb[c];
                    x = S.off[j] + S.size[j];
                }
                bool fits = true;
                int64_t gap_end = INT64_MAX;  // lowest neighbour start at or above x
                // neighbours 64 at a time: lane q holds neighbour e0 + q, read
                // by every lane with readlane
                for (int e0 = 0; e0 < m; e0 += kWave) {
                    int64_t oq = 0, eq = 0;
                    if (e0 + lane < m) {
                        const int j = S.nb[e0 + lane];
                        oq = S.off[j];
                        eq = oq + S.size[j];
                    }
                    const int cnt = min(kWave, m - e0);
                    for (int q = 0; q < cnt; ++q) {
                        const int64_t o = readlane64(oq, q), e = readlane64(eq, q);
                        if (x < e && o < x + st) fits = false;
                        if (o >= x && o < gap_end) gap_end = o;
                    }
                }
                if (c > m || !fits) continue;
                const uint64_t a0 = policy == MP_BEST_FIT
                                        ? (gap_end == INT64_MAX ? ~0ull : (uint64_t)(gap_end - x))
                                        : (uint64_t)x;
                const uint64_t a1 = policy == MP_BEST_FIT ? (uint64_t)x : 0ull;
                if (a0 < key0 || (a0 == key0 && a1 < key1)) {
                    key0 = a0;
                    key1 = a1;
                }
            }
            wave_min2(key0, key1);
            const int64_t x = policy == MP_BEST_FIT ? (int64_t)key1 : (int64_t)key0;
            if (lane == 0) {
                S.off[t] = x;
                S.n_nb = 0;
            }
            peak = max(peak, x + st);
        }
        __syncthreads();
    }
    if (tid < kWave) {
        for (int i = lane; i < n; i += kWave) offset_out[b0 + i] = S.off[i];
        if (lane == 0) peak_out[blockIdx.x] = peak;
    }
}

}  // namespace

hipError_t launch_breadth(const int64_t* begin, int64_t n_traces, const int32_t* num_ops,
                          const int64_t* size, const int32_t* first, const int32_t* last,
                          int64_t n_tensors, int32_t policy, int64_t* offset_out,
                          int64_t* peak_out, int32_t* status, hipStream_t st) {
    if (n_traces == 0) return hipSuccess;
    hipLaunchKernelGGL(breadth_kernel, dim3((unsigned)n_traces), dim3(kBBlock), 0, st, begin,
                       num_ops, size, first, last, n_tensors, policy, offset_out, peak_out,
                       status);
    return hipGetLastError();
}

}  // namespace mp
