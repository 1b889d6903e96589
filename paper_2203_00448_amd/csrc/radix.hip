// Stable LSD radix sort of (u64 key, u32 value) pairs, 8-bit digits:
// per-tile digit counts -> one device-wide exclusive scan in digit-major
// order -> stable scatter.  Inside a tile, elements are taken in rounds of
// 256 consecutive elements; a wave ranks equal digits with eight ballots and
// waves are ordered through per-(wave, digit) counts in LDS.  Up to 4,096
// pairs are sorted by one workgroup in LDS instead, in one launch.
#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr int kRadixBlock = 256;
constexpr int kRadixItems = 8;
constexpr int64_t kRadixTile = (int64_t)kRadixBlock * kRadixItems;
constexpr int kDigits = 256;

__global__ __launch_bounds__(kRadixBlock) void radix_count_kernel(const uint64_t* __restrict__ keys,
                                                                  int64_t n, int shift,
                                                                  int64_t* __restrict__ counts,
                                                                  int64_t n_tiles,
                                                                  const uint32_t* skip,
                                                                  const int64_t* n_live) {
    __shared__ uint32_t hist[kDigits];
    if (skip && *skip) return;
    if (n_live) n = min(n, *n_live);
    const int64_t base = (int64_t)blockIdx.x * kRadixTile;
    if (base >= n) {  // a tile past the live elements counts nothing
        counts[(int64_t)threadIdx.x * n_tiles + blockIdx.x] = 0;
        return;
    }
    hist[threadIdx.x] = 0;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kRadixItems; ++k) {
        const int64_t e = base + k * kRadixBlock + threadIdx.x;
        if (e < n) atomicAdd(&hist[(keys[e] >> shift) & 0xFF], 1u);
    }
    __syncthreads();
    counts[(int64_t)threadIdx.x * n_tiles + blockIdx.x] = hist[threadIdx.x];
}

__global__ __launch_bounds__(kRadixBlock) void radix_scatter_kernel(
    const uint64_t* __restrict__ kin, const uint32_t* __restrict__ vin, uint64_t* __restrict__ kout,
    uint32_t* __restrict__ vout, int64_t n, int shift, const int64_t* __restrict__ offs,
    int64_t n_tiles, const uint32_t* skip, const int64_t* n_live) {
    constexpr int kWaves = kRadixBlock / kWave;
    if (skip && *skip) return;
    if (n_live) n = min(n, *n_live);
    if ((int64_t)blockIdx.x * kRadixTile >= n) return;
    __shared__ uint32_t wave_cnt[kWaves][kDigits];
    __shared__ uint32_t running[kDigits];
    __shared__ int64_t gbase[kDigits];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    gbase[tid] = offs[(int64_t)tid * n_tiles + blockIdx.x];
    running[tid] = 0;
    const uint64_t lower = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    const int64_t base = (int64_t)blockIdx.x * kRadixTile;
    for (int k = 0; k < kRadixItems; ++k) {
        const int64_t e = base + k * kRadixBlock + tid;
        const bool valid = e < n;
        const uint64_t key = valid ? kin[e] : 0ull;
        const uint32_t val = (valid && vin) ? vin[e] : 0u;
        const uint32_t d = (uint32_t)((key >> shift) & 0xFF);
        uint64_t same = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
            const uint64_t ones = __ballot((d >> bit) & 1u);
            same &= ((d >> bit) & 1u) ? ones : ~ones;
        }
        const uint32_t rank = (uint32_t)__popcll(same & lower);
#pragma unroll
        for (int w = 0; w < kWaves; ++w) wave_cnt[w][tid] = 0;
        __syncthreads();
        if (valid && rank == 0) wave_cnt[wid][d] = (uint32_t)__popcll(same);
        __syncthreads();
        {  // digit tid: bases of each wave's group after all earlier elements
            uint32_t s = running[tid];
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                const uint32_t c = wave_cnt[w][tid];
                wave_cnt[w][tid] = s;
                s += c;
            }
            running[tid] = s;
        }
        __syncthreads();
        if (valid) {
            const int64_t pos = gbase[d] + wave_cnt[wid][d] + rank;
            kout[pos] = key;
            if (vout) vout[pos] = val;
        }
        __syncthreads();
    }
}

// One workgroup sorts up to kSmallSort pairs in LDS with a bitonic network
// over (the key's digit bits, input position).  Position breaks every tie, so
// the permutation is the one the stable digit passes produce; the pairs are
// written to the buffer those passes would end in (possibly the input: every
// input is in LDS before anything is written).  Elements [m, P) are padding
// that sorts last (all-ones key, position >= m).
constexpr int kSmallSort = 4096;
constexpr int kSmallSortThreads = 1024;

__global__ __launch_bounds__(kSmallSortThreads) void small_sort_kernel(
    const uint64_t* kin, const uint32_t* vin, uint64_t* kout, uint32_t* vout, int64_t n,
    int shift, uint64_t mask, int P, const uint32_t* skip, const int64_t* n_live) {
    __shared__ uint64_t sk[kSmallSort];  // full keys, moved by the network
    __shared__ uint16_t si[kSmallSort];  // input positions, moved with them
    __shared__ uint32_t sv[kSmallSort];  // values, by input position
    if (skip && *skip) return;
    int64_t m = n;
    if (n_live) m = min(m, *n_live);
    if (m < 0) m = 0;
    const int T = (int)blockDim.x, tid = (int)threadIdx.x;
    for (int i = tid; i < P; i += T) {
        const bool in = i < m;
        sk[i] = in ? kin[i] : ~0ull;
        si[i] = (uint16_t)i;
        if (vin) sv[i] = in ? vin[i] : 0u;
    }
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int t = tid; t < P / 2; t += T) {
                const int a = 2 * t - (t & (j - 1)), b = a + j;  // bit j of a clear
                const uint64_t ka = sk[a], kb = sk[b];
                const uint16_t ia = si[a], ib = si[b];
                const uint64_t da = (ka >> shift) & mask, db = (kb >> shift) & mask;
                const bool gt = da > db || (da == db && ia > ib);
                if (gt == ((a & k) == 0)) {  // ascending where bit k of a is clear
                    sk[a] = kb;
                    sk[b] = ka;
                    si[a] = ib;
                    si[b] = ia;
                }
            }
            __syncthreads();
        }
    }
    for (int r = tid; r < m; r += T) {
        kout[r] = sk[r];
        if (vout) vout[r] = sv[si[r]];
    }
}

}  // namespace

size_t radix_workspace_bytes(int64_t n) {
    const int64_t tiles = (n + kRadixTile - 1) / kRadixTile;
    const int64_t counts = tiles * kDigits;
    return (size_t)counts * sizeof(int64_t) + scan_workspace_bytes(counts);
}

// Sorts n pairs by bits [begin_bit, end_bit) of the key (in whole 8-bit
// digits), stably.  Buffers alternate between (k0, v0) and (k1, v1) once per
// digit; *in_alt tells where the result is (the single-workgroup sort of up
// to 4,096 pairs writes it there too).  v0/v1 may be null (keys only).  `ws` has radix_workspace_bytes(n).
// A non-null `skip` word that is nonzero at run time turns every kernel into
// a no-op (the buffers then stay as they were).  A non-null `n_live` is a
// device count read at run time: only the first min(n, *n_live) pairs are
// sorted (n then only bounds the launch).
hipError_t radix_sort_pairs(uint64_t* k0, uint32_t* v0, uint64_t* k1, uint32_t* v1, int64_t n,
                            int begin_bit, int end_bit, void* ws, bool* in_alt, hipStream_t st,
                            const uint32_t* skip, const int64_t* n_live) {
    *in_alt = false;
    if (n <= 1 || end_bit <= begin_bit) return hipSuccess;
    if (n <= kSmallSort) {
        const int passes = (end_bit - begin_bit + 7) / 8;
        const int width = min(8 * passes, 64 - begin_bit);  // the bits the passes order by
        const uint64_t mask = width >= 64 ? ~0ull : ((1ull << width) - 1ull);
        int P = 2;
        while (P < n) P <<= 1;
        const int threads = max(kWave, min(kSmallSortThreads, P / 2));
        const bool alt = (passes & 1) != 0;
        hipLaunchKernelGGL(small_sort_kernel, dim3(1), dim3(threads), 0, st, k0, v0,
                           alt ? k1 : k0, alt ? v1 : v0, n, begin_bit, mask, P, skip, n_live);
        *in_alt = alt;
        return hipGetLastError();
    }
    const int64_t tiles = (n + kRadixTile - 1) / kRadixTile;
    if (tiles > INT32_MAX) return hipErrorInvalidValue;
    int64_t* counts = static_cast<int64_t*>(ws);
    int64_t* partial = counts + tiles * kDigits;
    bool alt = false;
    for (int shift = begin_bit; shift < end_bit; shift += 8) {
        const uint64_t* ki = alt ? k1 : k0;
        const uint32_t* vi = alt ? v1 : v0;
        uint64_t* ko = alt ? k0 : k1;
        uint32_t* vo = alt ? v0 : v1;
        hipLaunchKernelGGL(radix_count_kernel, dim3((unsigned)tiles), dim3(kRadixBlock), 0, st, ki,
                           n, shift, counts, tiles, skip, n_live);
        hipError_t e = device_scan_i64(counts, tiles * kDigits, false, partial, nullptr, st, skip);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(radix_scatter_kernel, dim3((unsigned)tiles), dim3(kRadixBlock), 0, st,
                           ki, vi, ko, vo, n, shift, (const int64_t*)counts, tiles, skip,
                           n_live);
        alt = !alt;
    }
    *in_alt = alt;
    return hipGetLastError();
}

}  // namespace mp
