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
// workspace; within an op the words of all its tensors are spread over the
// workgroup's threads.  Writes are device-scope atomic maxima and the checks
// device-scope loads, so no stale cached line can hide an overwrite.  All
// checks of an op come before any of its clears, as in the definition above,
// also when its tensors are staged in several chunks.
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

// Barrier between phases that pass data through global memory.  The slab and
// the counting-sort arrays are written by plain stores and by atomics, both
// performed in L2, and read by loads that skip the L1; a workgroup barrier
// alone lets a wave pass while its stores are still on the way to L2, so a
// late clear could land after the next op's atomic maximum.  Each thread
// therefore first waits until all of its memory operations are complete.
__device__ __forceinline__ void l2_barrier() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
}

__global__ __launch_bounds__(kPBlock) void probe_kernel(
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, const int64_t* __restrict__ offset, int64_t n,
    int32_t num_ops, uint32_t* slab, int64_t slab_words, uint8_t* __restrict__ clob,
    int64_t* __restrict__ n_clob, int32_t* bstart, int32_t* dstart, int32_t* born, int32_t* dies,
    int32_t* __restrict__ status) {
    __shared__ uint64_t red[kPWaves];
    __shared__ int32_t carry;
    const int tid = threadIdx.x;

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
    l2_barrier();

    // ---- tensors by first and by last op (counting sort): counts, running
    // sums (bstart[t] = tensors first used before op t), then a scatter that
    // leaves bstart[t] at the end of op t's list
    for (int64_t i = tid; i < n; i += kPBlock) {
        atomicAdd(&bstart[first[i] + 1], 1);
        atomicAdd(&dstart[last[i] + 1], 1);
    }
    l2_barrier();
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
            l2_barrier();
        }
    }
    for (int64_t i = tid; i < n; i += kPBlock) {
        born[atomicAdd(&bstart[first[i]], 1)] = (int32_t)i;
        dies[atomicAdd(&dstart[last[i]], 1)] = (int32_t)i;
    }
    l2_barrier();

    // ---- replay.  An op's births, then its deaths, are staged in LDS (up to
    // kPBlock at a time) with an exclusive prefix of their word counts; all
    // threads then walk the concatenated words, word j by thread j % kPBlock,
    // so neighbouring lanes touch neighbouring words and a large tensor is
    // spread over the whole workgroup.
    __shared__ uint64_t s_pre[kPBlock + 1];  // first concatenated word of each entry
    __shared__ uint64_t s_w0[kPBlock];       // its first slab word
    __shared__ int32_t s_id[kPBlock];
    auto stage = [&](const int32_t* list, int32_t e0, int32_t e1) {  // returns the word total
        const int32_t e = e0 + tid;
        const bool has = e < e1;
        const int32_t i = has ? l2_load(&list[e]) : 0;
        const uint64_t wc = has ? (uint64_t)(size[i] >> 2) : 0;
        uint64_t tot;
        const uint64_t ex = block_exclusive_sum<kPBlock>(wc, &tot, red);
        s_pre[tid] = ex;
        s_w0[tid] = has ? (uint64_t)(offset[i] >> 2) : 0;
        s_id[tid] = i;
        if (tid == 0) s_pre[kPBlock] = ~0ull;
        __syncthreads();
        return tot;
    };
    // the entry holding concatenated word j (m entries, s_pre ascending)
    auto entry_of = [&](uint64_t j, int m) {
        int a = 0, z = m - 1;
        while (a < z) {
            const int mid = (a + z + 1) >> 1;
            if (s_pre[mid] <= j) a = mid;
            else z = mid - 1;
        }
        return a;
    };
    // walks over the staged words: atomic maxima, checks, clears
    auto write = [&](uint64_t tot, int m) {
        if (tid >= tot) return;
        int e = entry_of(tid, m);
        for (uint64_t j = tid; j < tot; j += kPBlock) {
            while (s_pre[e + 1] <= j) ++e;
            atomicMax(&slab[s_w0[e] + (j - s_pre[e])], (uint32_t)s_id[e] + 1u);
        }
    };
    auto check = [&](uint64_t tot, int m) {
        if (tid >= tot) return;
        int e = entry_of(tid, m);
        for (uint64_t j = tid; j < tot; j += 4 * kPBlock) {  // four loads in flight
            int ee[4];
            uint32_t got[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint64_t ju = j + (uint64_t)u * kPBlock;
                if (ju < tot) {
                    while (s_pre[e + 1] <= ju) ++e;
                    ee[u] = e;
                    got[u] = slab_load(&slab[s_w0[e] + (ju - s_pre[e])]);
                } else {
                    ee[u] = -1;
                    got[u] = 0;
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (ee[u] >= 0 && got[u] != (uint32_t)s_id[ee[u]] + 1u) clob[s_id[ee[u]]] = 1;
        }
    };
    auto clear = [&](uint64_t tot, int m) {
        if (tid >= tot) return;
        int e = entry_of(tid, m);
        for (uint64_t j = tid; j < tot; j += kPBlock) {
            while (s_pre[e + 1] <= j) ++e;
            slab[s_w0[e] + (j - s_pre[e])] = 0;
        }
    };
    for (int32_t t = 0; t < num_ops; ++t) {
        const int32_t b0 = t ? l2_load(&bstart[t - 1]) : 0, b1 = l2_load(&bstart[t]);
        const int32_t d0 = t ? l2_load(&dstart[t - 1]) : 0, d1 = l2_load(&dstart[t]);
        for (int32_t c0 = b0; c0 < b1; c0 += kPBlock) {
            write(stage(born, c0, b1), min(kPBlock, b1 - c0));
            l2_barrier();
        }
        // every check of op t before any of its clears; one chunk is staged
        // once, several are staged again for the clears
        const bool one = d1 - d0 <= kPBlock;
        for (int32_t c0 = d0; c0 < d1; c0 += kPBlock) {
            const int m = min(kPBlock, d1 - c0);
            const uint64_t tot = stage(dies, c0, d1);
            check(tot, m);
            __syncthreads();
            if (one) clear(tot, m);
        }
        if (!one)
            for (int32_t c0 = d0; c0 < d1; c0 += kPBlock) {
                clear(stage(dies, c0, d1), min(kPBlock, d1 - c0));
                __syncthreads();
            }
        if (d1 > d0) l2_barrier();
    }
    uint64_t hits = 0;
    for (int64_t i = tid; i < n; i += kPBlock) hits += clob[i];
    hits = block_reduce<kPBlock>(hits, OpAdd<uint64_t>(), red);
    if (tid == 0) *n_clob = (int64_t)hits;
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
