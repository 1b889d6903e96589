// Device-side helpers shared by the planner kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "memoplan.h"

namespace mp {

constexpr int kWave = 64;
constexpr uint32_t kUnplaced = 0xFFFFFFFFu;

__device__ __forceinline__ void raise_status(int32_t* status, int32_t code) {
    if (code != MP_OK) atomicMin(status, code);
}

// LDS words that other waves of the workgroup poll.
__device__ __forceinline__ uint32_t lds_poll(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_publish(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Saturating unsigned 64-bit add (associative, so any reduction order agrees).
__device__ __forceinline__ uint64_t sat_add(uint64_t a, uint64_t b) {
    uint64_t s = a + b;
    return s < a ? ~0ull : s;
}

template <typename T>
struct OpMax {
    __device__ T operator()(T a, T b) const { return a > b ? a : b; }
};
template <typename T>
struct OpMin {
    __device__ T operator()(T a, T b) const { return a < b ? a : b; }
};
template <typename T>
struct OpOr {
    __device__ T operator()(T a, T b) const { return a | b; }
};
template <typename T>
struct OpAdd {
    __device__ T operator()(T a, T b) const { return a + b; }
};
struct OpSatAdd {
    __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return sat_add(a, b); }
};

template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v = op(v, __shfl_xor(v, o, kWave));
    return v;
}

// Reduction over the whole workgroup; every thread gets the result.
// `scratch` holds BLOCK / 64 values.  Contains two barriers.
template <int BLOCK, typename T, typename Op>
__device__ __forceinline__ T block_reduce(T v, Op op, T* scratch) {
    v = wave_reduce(v, op);
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    if (lane == 0) scratch[wid] = v;
    __syncthreads();
    T r = scratch[0];
#pragma unroll
    for (int w = 1; w < BLOCK / kWave; ++w) r = op(r, scratch[w]);
    __syncthreads();
    return r;
}

// Inclusive prefix sum across the 64 lanes of a wave (unsigned 32 or 64 bit).
template <typename T>
__device__ __forceinline__ T wave_inclusive_sum(T x) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        T y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    return x;
}

// Exclusive prefix of one value per thread over the workgroup (thread order);
// returns the prefix, *total gets the sum.  `scratch` holds BLOCK/64 values.
// Contains two barriers.
template <int BLOCK, typename T>
__device__ __forceinline__ T block_exclusive_sum(T v, T* total, T* scratch) {
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    T inc = wave_inclusive_sum(v);
    if (lane == kWave - 1) scratch[wid] = inc;
    __syncthreads();
    T before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < BLOCK / kWave; ++w) {
        T t = scratch[w];
        before += (w < wid) ? t : T(0);
        all += t;
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

}  // namespace mp
