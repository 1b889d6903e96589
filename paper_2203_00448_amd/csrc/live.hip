// Live-bytes profile of one trace: live[t] = sum of the sizes of the tensors
// alive at op t (first <= t <= last), and its maximum -- a lower bound on the
// arena size of any valid plan, since every tensor alive at t needs its own
// bytes.  Difference array with 64-bit atomics (+size at first, -size at
// last + 1), then an inclusive device-wide prefix sum.
#include <mutex>

#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr int kLiveBlock = 256;

__global__ void live_init_kernel(int64_t* __restrict__ live, int32_t num_ops,
                                 int64_t* __restrict__ max_out, uint64_t* __restrict__ sum) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < num_ops; t += stride)
        live[t] = 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        *max_out = 0;
        *sum = 0;
    }
}

__global__ __launch_bounds__(kLiveBlock) void live_delta_kernel(
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, int64_t n, int32_t num_ops, int64_t* __restrict__ live,
    uint64_t* __restrict__ sum, int32_t* __restrict__ status) {
    __shared__ uint64_t red[kLiveBlock / kWave];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    uint32_t bad = 0;
    uint64_t acc = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int64_t s = size[i];
        const int32_t f = first[i], l = last[i];
        if (s <= 0 || f < 0 || f > l || l >= num_ops) {
            bad = 1;
            if (s > 0) acc = sat_add(acc, (uint64_t)s);
            continue;  // no writes for a tensor outside the op range
        }
        acc = sat_add(acc, (uint64_t)s);
        atomicAdd(reinterpret_cast<unsigned long long*>(live + f), (unsigned long long)s);
        if (l + 1 < num_ops)
            atomicAdd(reinterpret_cast<unsigned long long*>(live + l + 1),
                      (unsigned long long)(-s));
    }
    bad = block_reduce<kLiveBlock>(bad, OpOr<uint32_t>(), reinterpret_cast<uint32_t*>(red));
    acc = block_reduce<kLiveBlock>(acc, OpSatAdd(), red);
    if (threadIdx.x == 0) {
        if (bad) raise_status(status, MP_EINVAL);
        // global saturating sum: once past INT64_MAX the overflow is reported
        const uint64_t old = atomicAdd(reinterpret_cast<unsigned long long*>(sum),
                                       (unsigned long long)acc);
        if (acc > (uint64_t)INT64_MAX || old > (uint64_t)INT64_MAX - acc)
            raise_status(status, MP_EOVERFLOW);
    }
}

}  // namespace

size_t live_workspace_bytes(int32_t num_ops) {
    return 256 + scan_workspace_bytes(num_ops > 0 ? num_ops : 1);
}

hipError_t launch_live_profile(const int64_t* size, const int32_t* first, const int32_t* last,
                               int64_t n, int32_t num_ops, int64_t* live_out, int64_t* max_out,
                               void* ws, int32_t* status, hipStream_t st) {
    uint64_t* sum = static_cast<uint64_t*>(ws);
    int64_t* partial = reinterpret_cast<int64_t*>(static_cast<char*>(ws) + 256);
    const int64_t ig = ((int64_t)num_ops + 255) / 256 + 1;
    const unsigned init_grid = (unsigned)(ig < 1024 ? ig : 1024);
    hipLaunchKernelGGL(live_init_kernel, dim3(init_grid), dim3(256), 0, st, live_out, num_ops,
                       max_out, sum);
    if (n > 0) {
        const int64_t g = (n + kLiveBlock - 1) / kLiveBlock;
        const unsigned grid = (unsigned)(g < 2048 ? g : 2048);
        hipLaunchKernelGGL(live_delta_kernel, dim3(grid), dim3(kLiveBlock), 0, st, size, first,
                           last, n, num_ops, live_out, sum, status);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return device_scan_i64(live_out, num_ops, true, partial,
                           reinterpret_cast<unsigned long long*>(max_out), st);
}

// ---- the same profile without a caller workspace (no allocation anywhere)
//
// Scratch of mp_live_bytes_profile_noalloc: the running-sum word and the
// scan's tile partials, for at most MP_LIVE_NOALLOC_MAX_OPS ops.  Each GPU
// the library runs on holds one copy until the process ends; every call on a
// GPU shares it.  Host code never passes `scratch` itself to a kernel (on the
// host it is only a stand-in for the symbol): the device address is looked up
// once per device with that device current and kept in scratch_ptr.
namespace {

constexpr size_t kNoallocScratchBytes = 256 + ((size_t)MP_LIVE_NOALLOC_MAX_OPS / 2048 + 2) * 8;
__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of this device's scratch (looked up on first use), or
// nullptr if it cannot be resolved.
void* scratch_ptr() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

size_t live_noalloc_scratch_bytes() { return kNoallocScratchBytes; }

hipError_t launch_live_profile_noalloc(const int64_t* size, const int32_t* first,
                                       const int32_t* last, int64_t n, int32_t num_ops,
                                       int64_t* live_out, int64_t* max_out, int32_t* status,
                                       hipStream_t st) {
    static_assert(kNoallocScratchBytes >= 256 + (MP_LIVE_NOALLOC_MAX_OPS + 2047) / 2048 * 8 + 8,
                  "scratch holds the sum word and every tile partial");
    if (num_ops < 0 || live_workspace_bytes(num_ops) > kNoallocScratchBytes)
        return hipErrorInvalidValue;
    void* ws = scratch_ptr();
    if (!ws) return hipErrorInvalidSymbol;
    return launch_live_profile(size, first, last, n, num_ops, live_out, max_out, ws, status, st);
}

}  // namespace mp
