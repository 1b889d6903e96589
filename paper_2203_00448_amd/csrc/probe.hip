// Write-pattern aliasing probe of a plan.
//
// Section 3.3 applies a plan by allocating one slab of total_size bytes and
// placing every tensor as a view at its offset (Listing 5).  The probe
// exercises such a slab the way execution would: the ops of the trace are
// replayed in order over the slab seen as 32-bit words, zero at the start.
// At op t every tensor first used at t writes id + 1 into each word of its
// byte range, keeping the larger value where a word already holds one (so
// the writers of one op resolve the same way in any order); then every
// tensor last used at t checks each word of its range -- a tensor that finds
// another value is "clobbered" -- and then clears its words to 0.  A valid
// plan clobbers nothing; of every pair that breaks the constraints of Eq. 2.1
// at least one member is clobbered.
//
// One workgroup replays the whole trace: ops are sequential by definition.
// Tensors are listed by first and by last op with a counting sort in the
// workspace; within an op, a wave takes a tensor and its lanes stride over
// the tensor's words.  Ops without a last use cost no barrier.  Writes are
// device-scope atomic maxima and the checks device-scope loads, so no stale
// cached line can hide an overwrite.
#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr int kPBlock = 1024;
constexpr int kPWaves = kPBlock / kWave;

// Reads of words that atomics wrote (performed in L2) go to L2 as well.
__device__ __forceinline__ uint32_t slab_load(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t l2_load(const int32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kPBlock) void probe_kernel(
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, const int64_t* __restrict__ offset, int64_t n,
    int32_t num_ops, uint32_t* slab, int64_t slab_words, uint8_t* __restrict__ clob,
    int64_t* __restrict__ n_clob, int32_t* bstart, int32_t* dstart, int32_t* born, int32_t* dies,
    int32_t* __restrict__ status) {
    __shared__ uint64_t red[kPWaves];
    __shared__ int32_t carry;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;

    // ---- checks, and the highest word the plan touches
    uint64_t bad = 0, top = 0;
    for (int64_t i = tid; i < n; i += kPBlock) {
        const int64_t s = size[i], o = offset[i];
        const int32_t f = first[i], l = last[i];
        if (s <= 0 || (s & 3) || o < 0 || (o & 3) || o > INT64_MAX - s || f < 0 || f > l ||
            l >= num_ops)
            bad = 1;
        else
            top = max(top, (uint64_t)((o + s) >> 2));
    }
    bad = block_reduce<kPBlock>(bad, OpMax<uint64_t>(), red);
    top = block_reduce<kPBlock>(top, OpMax<uint64_t>(), red);
    if (bad || top > (uint64_t)slab_words) {
        if (tid == 0) raise_status(status, MP_EINVAL);
        return;
    }

    // ---- zeroed slab, outputs and op counters
    for (int64_t w = tid; w < (int64_t)top; w += kPBlock) slab[w] = 0;
    for (int64_t i = tid; i < n; i += kPBlock) clob[i] = 0;
    for (int32_t t = tid; t <= num_ops; t += kPBlock) {
        bstart[t] = 0;
        dstart[t] = 0;
    }
    __syncthreads();

    // ---- tensors by first and by last op (counting sort): counts, running
    // sums (bstart[t] = tensors first used before op t), then a scatter that
    // leaves bstart[t] at the end of op t's list
    for (int64_t i = tid; i < n; i += kPBlock) {
        atomicAdd(&bstart[first[i] + 1], 1);
        atomicAdd(&dstart[last[i] + 1], 1);
    }
    __syncthreads();
    for (int h = 0; h < 2; ++h) {
        int32_t* c = h ? dstart : bstart;
        if (tid == 0) carry = 0;
        __syncthreads();
        for (int32_t base = 0; base <= num_ops; base += kPBlock) {
            const int32_t t = base + tid;
            const int32_t v = t <= num_ops ? l2_load(&c[t]) : 0;
            int32_t tot;
            const int32_t ex = block_exclusive_sum<kPBlock>(v, &tot, reinterpret_cast<int32_t*>(red));
            if (t <= num_ops) c[t] = carry + ex + v;
            __syncthreads();
            if (tid == 0) carry += tot;
            __syncthreads();
        }
    }
    for (int64_t i = tid; i < n; i += kPBlock) {
        born[atomicAdd(&bstart[first[i]], 1)] = (int32_t)i;
        dies[atomicAdd(&dstart[last[i]], 1)] = (int32_t)i;
    }
    __syncthreads();

    // ---- replay
    int64_t hits = 0;
    for (int32_t t = 0; t < num_ops; ++t) {
        const int32_t b0 = t ? l2_load(&bstart[t - 1]) : 0, b1 = l2_load(&bstart[t]);
        const int32_t d0 = t ? l2_load(&dstart[t - 1]) : 0, d1 = l2_load(&dstart[t]);
        for (int32_t k = b0 + wid; k < b1; k += kPWaves) {  // writes: a wave per tensor
            const int32_t i = l2_load(&born[k]);
            const uint32_t v = (uint32_t)i + 1u;
            const int64_t w0 = offset[i] >> 2, w1 = (offset[i] + size[i]) >> 2;
            for (int64_t w = w0 + lane; w < w1; w += kWave) atomicMax(&slab[w], v);
        }
        if (d0 == d1) continue;
        __syncthreads();
        for (int32_t k = d0 + wid; k < d1; k += kPWaves) {  // checks
            const int32_t i = l2_load(&dies[k]);
            const uint32_t v = (uint32_t)i + 1u;
            const int64_t w0 = offset[i] >> 2, w1 = (offset[i] + size[i]) >> 2;
            bool foreign = false;
            for (int64_t w = w0 + lane; w < w1; w += kWave) foreign |= slab_load(&slab[w]) != v;
            if (__ballot(foreign) && lane == 0) {
                clob[i] = 1;
                ++hits;
            }
        }
        __syncthreads();
        for (int32_t k = d0 + wid; k < d1; k += kPWaves) {  // clears
            const int32_t i = l2_load(&dies[k]);
            const int64_t w0 = offset[i] >> 2, w1 = (offset[i] + size[i]) >> 2;
            for (int64_t w = w0 + lane; w < w1; w += kWave) slab[w] = 0;
        }
        __syncthreads();
    }
    hits = block_reduce<kPBlock>((uint64_t)hits, OpAdd<uint64_t>(), red);
    if (tid == 0) *n_clob = hits;
}

}  // namespace

size_t probe_workspace_bytes(int64_t n, int32_t num_ops) {
    if (n < 0 || n >= INT32_MAX || num_ops < 0) return 0;
    return (2 * ((size_t)num_ops + 1) + 2 * (size_t)(n > 0 ? n : 1)) * sizeof(int32_t);
}

hipError_t launch_probe(const int64_t* size, const int32_t* first, const int32_t* last,
                        const int64_t* offset, int64_t n, int32_t num_ops, void* slab,
                        size_t slab_bytes, uint8_t* clob, int64_t* n_clob, void* ws,
                        int32_t* status, hipStream_t st) {
    int32_t* b = static_cast<int32_t*>(ws);
    int32_t* d = b + (num_ops + 1);
    int32_t* born = d + (num_ops + 1);
    int32_t* dies = born + (n > 0 ? n : 1);
    hipLaunchKernelGGL(probe_kernel, dim3(1), dim3(kPBlock), 0, st, size, first, last, offset, n,
                       num_ops, static_cast<uint32_t*>(slab), (int64_t)(slab_bytes / 4), clob,
                       n_clob, b, d, born, dies, status);
    return hipGetLastError();
}

}  // namespace mp
