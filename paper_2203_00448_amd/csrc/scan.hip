// Device-wide prefix sums over int64 arrays (reduce, scan of tile totals,
// rescan), used by the liveness profile and by plan validation.
#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr int kScanBlock = 256;
constexpr int kScanItems = 8;
constexpr int64_t kScanTile = (int64_t)kScanBlock * kScanItems;

__device__ __forceinline__ int64_t wave_inclusive_sum64(int64_t x) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int64_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    return x;
}

// Exclusive prefix of one value per thread over the workgroup.
template <int BLOCK>
__device__ __forceinline__ int64_t block_exclusive_sum64(int64_t v, int64_t* total,
                                                         int64_t* scratch) {
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    const int64_t inc = wave_inclusive_sum64(v);
    if (lane == kWave - 1) scratch[wid] = inc;
    __syncthreads();
    int64_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < BLOCK / kWave; ++w) {
        const int64_t t = scratch[w];
        before += (w < wid) ? t : 0;
        all += t;
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

__global__ __launch_bounds__(kScanBlock) void tile_sums_kernel(const int64_t* __restrict__ data,
                                                               int64_t n,
                                                               int64_t* __restrict__ partial,
                                                               const uint32_t* skip) {
    __shared__ int64_t scratch[kScanBlock / kWave];
    if (skip && *skip) return;
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k)
        if (base + k < n) s += data[base + k];
    int64_t total;
    block_exclusive_sum64<kScanBlock>(s, &total, scratch);
    if (threadIdx.x == 0) partial[blockIdx.x] = total;
}

// One workgroup: exclusive scan of partial[0..m) in place; partial[m] = total.
__global__ __launch_bounds__(1024) void scan_partials_kernel(int64_t* __restrict__ partial,
                                                             int64_t m, const uint32_t* skip) {
    __shared__ int64_t scratch[1024 / kWave];
    if (skip && *skip) return;
    int64_t carry = 0;
    for (int64_t base = 0; base < m; base += 1024 * kScanItems) {
        const int64_t i0 = base + (int64_t)threadIdx.x * kScanItems;
        int64_t v[kScanItems];
        int64_t s = 0;
#pragma unroll
        for (int k = 0; k < kScanItems; ++k) {
            v[k] = (i0 + k < m) ? partial[i0 + k] : 0;
            s += v[k];
        }
        int64_t total;
        int64_t run = carry + block_exclusive_sum64<1024>(s, &total, scratch);
#pragma unroll
        for (int k = 0; k < kScanItems; ++k) {
            if (i0 + k < m) partial[i0 + k] = run;
            run += v[k];
        }
        carry += total;
    }
    if (threadIdx.x == 0) partial[m] = carry;
}

__global__ __launch_bounds__(kScanBlock) void rescan_kernel(int64_t* __restrict__ data, int64_t n,
                                                            const int64_t* __restrict__ partial,
                                                            int inclusive,
                                                            unsigned long long* max_out,
                                                            const uint32_t* skip) {
    __shared__ int64_t scratch[kScanBlock / kWave];
    if (skip && *skip) return;
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int64_t v[kScanItems];
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = (base + k < n) ? data[base + k] : 0;
        s += v[k];
    }
    int64_t total;
    int64_t run = partial[blockIdx.x] + block_exclusive_sum64<kScanBlock>(s, &total, scratch);
    int64_t mx = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        if (base + k < n) {
            const int64_t out = inclusive ? run + v[k] : run;
            data[base + k] = out;
            mx = out > mx ? out : mx;
        }
        run += v[k];
    }
    if (max_out) {
        mx = wave_reduce(mx, OpMax<int64_t>());
        if ((threadIdx.x & (kWave - 1)) == 0 && mx > 0) atomicMax(max_out, (unsigned long long)mx);
    }
}

// Short arrays (up to kSmallScan values) in one launch: one workgroup of
// 1024 threads, 16 contiguous values a thread; partial[tiles] gets the total
// as after the three-kernel scan.
constexpr int kSmallBlock = 1024;
constexpr int kSmallItems = 16;
constexpr int64_t kSmallScan = (int64_t)kSmallBlock * kSmallItems;

__global__ __launch_bounds__(kSmallBlock) void scan_small_kernel(int64_t* __restrict__ data,
                                                                  int64_t n, int inclusive,
                                                                  int64_t* __restrict__ partial,
                                                                  int64_t tiles,
                                                                  unsigned long long* max_out,
                                                                  const uint32_t* skip) {
    __shared__ int64_t scratch[kSmallBlock / kWave];
    if (skip && *skip) return;
    const int64_t base = (int64_t)threadIdx.x * kSmallItems;
    int64_t v[kSmallItems];
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kSmallItems; ++k) {
        v[k] = (base + k < n) ? data[base + k] : 0;
        s += v[k];
    }
    int64_t total;
    int64_t run = block_exclusive_sum64<kSmallBlock>(s, &total, scratch);
    int64_t mx = 0;
#pragma unroll
    for (int k = 0; k < kSmallItems; ++k) {
        if (base + k < n) {
            const int64_t out = inclusive ? run + v[k] : run;
            data[base + k] = out;
            mx = out > mx ? out : mx;
        }
        run += v[k];
    }
    if (threadIdx.x == 0) partial[tiles] = total;
    if (max_out) {
        mx = wave_reduce(mx, OpMax<int64_t>());
        if ((threadIdx.x & (kWave - 1)) == 0 && mx > 0) atomicMax(max_out, (unsigned long long)mx);
    }
}

}  // namespace

size_t scan_workspace_bytes(int64_t n) {
    const int64_t tiles = (n + kScanTile - 1) / kScanTile;
    return (size_t)(tiles + 1) * sizeof(int64_t);
}

// In-place prefix sum of data[0..n): exclusive or inclusive.  `partial` is a
// workspace of scan_workspace_bytes(n); afterwards partial[tiles] holds the
// total.  If max_out is given, atomicMax of the (non-negative) results.
// With a non-null `skip` word that is nonzero when the kernels run, they do
// nothing (lets a caller enqueue a data-dependent optional step).
hipError_t device_scan_i64(int64_t* data, int64_t n, bool inclusive, int64_t* partial,
                           unsigned long long* max_out, hipStream_t st, const uint32_t* skip) {
    if (n <= 0) return hipSuccess;
    const int64_t tiles = (n + kScanTile - 1) / kScanTile;
    if (tiles > INT32_MAX) return hipErrorInvalidValue;
    if (n <= kSmallScan) {
        hipLaunchKernelGGL(scan_small_kernel, dim3(1), dim3(kSmallBlock), 0, st, data, n,
                           inclusive ? 1 : 0, partial, tiles, max_out, skip);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(tile_sums_kernel, dim3((unsigned)tiles), dim3(kScanBlock), 0, st, data, n,
                       partial, skip);
    hipLaunchKernelGGL(scan_partials_kernel, dim3(1), dim3(1024), 0, st, partial, tiles, skip);
    hipLaunchKernelGGL(rescan_kernel, dim3((unsigned)tiles), dim3(kScanBlock), 0, st, data, n,
                       (const int64_t*)partial, inclusive ? 1 : 0, max_out, skip);
    return hipGetLastError();
}

}  // namespace mp
