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
// What happens to a word depends only on the tensors whose ranges cover it,
// so the replay splits by address: the slab is cut into tiles of 64 words,
// one wave replays one tile with one word per lane, and only the events of
// the tensors covering the tile are visited, in op order (births before
// deaths).  The per-tile event lists are one radix sort of (tile, 2 op +
// kind) keys, one key per tensor, tile and kind.  A lane owns its word for
// the whole replay: it keeps the word's value in a register for the maxima,
// stores every change to the slab, and checks what it reads back from the
// slab.  The number of (tensor, tile) pairs is known only on the device;
// when it exceeds what the workspace holds, the tiled kernels stand down and
// one workgroup replays the ops one after another instead (same results).

#include <type_traits>

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

// Device words that choose the path of one call.
struct ProbeFlags {
    uint32_t bad;      // an input failed its checks
    uint32_t skip;     // the tiled kernels do nothing (bad input, or too many pairs)
    uint32_t run_ops;  // the op-by-op replay runs instead
    uint32_t pad;
    unsigned long long top;  // one past the highest word the plan touches
    int64_t n_tiles;         // tiles of 64 words below top
    uint32_t n_big;          // tensors over more than kSmallSpan tiles
    uint32_t sink;           // written by lanes past the top of the slab, never read
};
static_assert(sizeof(ProbeFlags) <= 256, "the flags fill the first 256 workspace bytes");

// ---------------------------------------------------------------------------
// Op-by-op replay: one workgroup walks the ops in order.  Tensors are listed
// by first and by last op with a counting sort in the workspace; within an op
// the words of all its tensors are spread over the workgroup's threads.
// Writes are device-scope atomic maxima and the checks device-scope loads, so
// no stale cached line can hide an overwrite.  All checks of an op come
// before any of its clears, also when its tensors are staged in chunks.
__global__ __launch_bounds__(kPBlock) void probe_ops_kernel(
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, const int64_t* __restrict__ offset, int64_t n,
    int32_t num_ops, uint32_t* slab, int64_t slab_words, uint8_t* __restrict__ clob,
    int64_t* __restrict__ n_clob, int32_t* bstart, int32_t* dstart, int32_t* born, int32_t* dies,
    int32_t* __restrict__ status, const ProbeFlags* fl) {
    __shared__ uint64_t red[kPWaves];
    __shared__ int32_t carry;
    const int tid = threadIdx.x;
    if (!fl->run_ops) return;

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

// ---------------------------------------------------------------------------
// Tiled replay.

constexpr int kTileShift = 6;  // 64 words (256 bytes) per tile, one per lane
constexpr int kTBlock = 256;
constexpr int kTWaves = kTBlock / kWave;
constexpr int kSmallSpan = 16;  // tensors over more tiles are emitted by whole workgroups
constexpr int kUnroll = 8;      // events whose checks are in flight together
constexpr int kPad = 2 * kUnroll;  // event-buffer entries past the capacity (read ahead)

__global__ void probe_init_kernel(ProbeFlags* fl, int64_t* n_clob) {
    fl->bad = 0;
    fl->skip = 1;
    fl->run_ops = 0;
    fl->pad = 0;
    fl->top = 0;
    fl->n_tiles = 0;
    fl->n_big = 0;
    *n_clob = 0;
}

// Checks every tensor, clears its flag and counts its events: a birth and a
// death in each tile its range meets.
__global__ __launch_bounds__(kTBlock) void probe_prepare_kernel(
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, const int64_t* __restrict__ offset, int64_t n,
    int32_t num_ops, uint8_t* __restrict__ clob, int64_t* __restrict__ cnt, ProbeFlags* fl) {
    const int64_t i = (int64_t)blockIdx.x * kTBlock + threadIdx.x;
    bool bad = false;
    uint64_t top = 0;
    if (i < n) {
        const int64_t s = size[i], o = offset[i];
        const int32_t f = first[i], l = last[i];
        if (s <= 0 || (s & 3) || o < 0 || (o & 3) || o > INT64_MAX - s || f < 0 || f > l ||
            l >= num_ops) {
            bad = true;
            cnt[i] = 0;
        } else {
            const uint64_t w0 = (uint64_t)o >> 2, w1 = (uint64_t)(o + s) >> 2;
            top = w1;
            cnt[i] = 2 * (int64_t)(((w1 - 1) >> kTileShift) - (w0 >> kTileShift) + 1);
        }
        clob[i] = 0;
    }
    if (__ballot(bad) && (threadIdx.x & (kWave - 1)) == 0) atomicOr(&fl->bad, 1u);
    __shared__ uint64_t red[kTWaves];
    top = block_reduce<kTBlock>(top, OpMax<uint64_t>(), red);
    if (threadIdx.x == 0 && top) atomicMax(&fl->top, (unsigned long long)top);
}

// Picks the path once the inputs are checked and the events are counted.
__global__ void probe_decide_kernel(ProbeFlags* fl, const int64_t* total, int64_t capacity,
                                    int64_t slab_words, int32_t* status) {
    if (fl->bad || fl->top > (unsigned long long)slab_words) {
        raise_status(status, MP_EINVAL);
        return;  // skip stays set, run_ops clear
    }
    fl->n_tiles = (int64_t)((fl->top + 63) >> kTileShift);
    const bool fits = *total <= capacity;
    fl->skip = fits ? 0u : 1u;
    fl->run_ops = fits ? 0u : 1u;
}

// Writes the events of each tensor at its place in the exclusive prefix of
// the counts: key (tile << op_bits) | (2 first) for the birth and
// (tile << op_bits) | (2 last + 1) for the death, value the tensor id.  A
// thread writes the events of a tensor over at most kSmallSpan tiles and
// lists the larger ones for probe_emit_big_kernel.
__device__ __forceinline__ void emit_pair(uint64_t* keys, uint32_t* vals, int64_t e, uint64_t t,
                                          int op_bits, uint64_t kb, uint64_t kd, uint32_t i) {
    keys[e] = (t << op_bits) | kb;
    vals[e] = i;
    keys[e + 1] = (t << op_bits) | kd;
    vals[e + 1] = i;
}

__global__ __launch_bounds__(kTBlock) void probe_emit_kernel(
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, const int64_t* __restrict__ offset, int64_t n, int op_bits,
    const int64_t* __restrict__ base, uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
    int32_t* __restrict__ big, ProbeFlags* fl) {
    if (fl->skip) return;
    const int64_t i = (int64_t)blockIdx.x * kTBlock + threadIdx.x;
    if (i >= n) return;
    const int64_t o = offset[i], s = size[i];
    const uint64_t t0 = ((uint64_t)o >> 2) >> kTileShift;
    const uint64_t t1 = (((uint64_t)(o + s) >> 2) - 1) >> kTileShift;
    if (t1 - t0 >= (uint64_t)kSmallSpan) {
        big[atomicAdd(&fl->n_big, 1u)] = (int32_t)i;
        return;
    }
    const uint64_t kb = 2ull * (uint32_t)first[i], kd = 2ull * (uint32_t)last[i] + 1;
    int64_t e = base[i];
    for (uint64_t t = t0; t <= t1; ++t, e += 2) emit_pair(keys, vals, e, t, op_bits, kb, kd, (uint32_t)i);
}

// One workgroup per listed tensor (grid-stride over the list).
__global__ __launch_bounds__(kTBlock) void probe_emit_big_kernel(
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, const int64_t* __restrict__ offset, int op_bits,
    const int64_t* __restrict__ base, uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
    const int32_t* __restrict__ big, const ProbeFlags* fl) {
    if (fl->skip) return;
    const uint32_t n_big = fl->n_big;
    for (uint32_t b = blockIdx.x; b < n_big; b += gridDim.x) {
        const int32_t i = big[b];
        const int64_t o = offset[i], s = size[i];
        const uint64_t t0 = ((uint64_t)o >> 2) >> kTileShift;
        const uint64_t t1 = (((uint64_t)(o + s) >> 2) - 1) >> kTileShift;
        const uint64_t kb = 2ull * (uint32_t)first[i], kd = 2ull * (uint32_t)last[i] + 1;
        const int64_t e0 = base[i];
        for (uint64_t t = t0 + threadIdx.x; t <= t1; t += kTBlock)
            emit_pair(keys, vals, e0 + 2 * (int64_t)(t - t0), t, op_bits, kb, kd, (uint32_t)i);
    }
}

// First index in [0, total) whose tile (key >> op_bits) is >= tile, or > tile
// when `after`; total if there is none.  The wave samples 64 evenly spaced
// keys per round, so a million keys take four rounds of one load each.
__device__ int64_t wave_find(const uint64_t* __restrict__ keys, int64_t total, int op_bits,
                             uint64_t tile, bool after, int lane) {
    int64_t lo = 0, hi = total;  // the answer lies in [lo, hi]; hi is total or a hit
    while (lo < hi) {
        const int64_t step = (hi - lo + kWave - 1) / kWave;
        const int64_t idx = lo + (int64_t)(lane + 1) * step - 1;
        bool hit = true;
        if (idx < hi) {
            const uint64_t t = keys[idx] >> op_bits;
            hit = after ? t > tile : t >= tile;
        }
        const uint64_t b = __ballot(hit);
        if (!b) return hi;
        const int f = __builtin_ctzll(b);
        hi = min(hi, lo + (int64_t)(f + 1) * step - 1);
        lo += (int64_t)f * step;
    }
    return lo;
}

// Packs each sorted event for the replay as four words, in the form the
// replay uses them: the mask of the lanes (words) of its tile that the tensor
// covers (two words); the tensor id + 1, with bit 31 set when the event starts
// a group -- a run of equal keys, the births or the deaths of one op in one
// tile; and all ones for a death, 0 for a birth.
__global__ __launch_bounds__(kTBlock) void probe_pack_kernel(
    const int64_t* __restrict__ size, const int64_t* __restrict__ offset,
    const uint64_t* __restrict__ keys, const uint32_t* __restrict__ vals,
    const int64_t* __restrict__ total_p, int op_bits, uint4* __restrict__ packed,
    const ProbeFlags* fl) {
    if (fl->skip) return;
    const int64_t total = *total_p;
    for (int64_t k = (int64_t)blockIdx.x * kTBlock + threadIdx.x; k < total;
         k += (int64_t)gridDim.x * kTBlock) {
        const uint64_t key = keys[k];
        const uint32_t id = vals[k];
        const bool start = k == 0 || keys[k - 1] != key;
        const int64_t tbase = (int64_t)(key >> op_bits) << kTileShift, o = offset[id];
        const int lo = (int)max((o >> 2) - tbase, (int64_t)0);                  // 0..63
        const int hi = (int)min(((o + size[id]) >> 2) - tbase, (int64_t)kWave);  // 1..64
        const uint64_t mask = (hi == kWave ? ~0ull : (1ull << hi) - 1) & ~((1ull << lo) - 1);
        packed[k] = make_uint4((uint32_t)mask, (uint32_t)(mask >> 32),
                               (id + 1u) | (start ? 1u << 31 : 0u), (key & 1u) ? ~0u : 0u);
    }
}

__device__ __forceinline__ uint32_t lane_word_load(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}
__device__ __forceinline__ void lane_word_store(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}

// A value the whole wave holds, moved to scalar registers.
__device__ __forceinline__ int64_t uniform64(int64_t x) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// kUnroll packed events read through the scalar cache (the index is the same
// for the whole wave), so they land in scalar registers.
struct EventGroup {
    uint32_t w[4 * kUnroll];
};
typedef const __attribute__((address_space(4))) uint32_t* ConstWords;
__device__ __forceinline__ EventGroup group_at(const uint4* packed, int64_t k) {
    const ConstWords p = (ConstWords)(packed + k);
    EventGroup g;
#pragma unroll
    for (int i = 0; i < 4 * kUnroll; ++i) g.w[i] = p[i];
    return g;
}
__device__ __forceinline__ uint64_t pair64(uint32_t lo, uint32_t hi) {
    return ((uint64_t)hi << 32) | lo;
}

// One wave per tile, word tile * 64 + lane per lane.  The slab accesses are
// relaxed atomics at wavefront scope only so that every change really goes
// to memory and every check really reads it back; no other lane ever touches
// the word.  Each event is: clear the word if the event starts a group and
// the previous group held deaths covering it; store the word (which also
// lands the previous event's write); read it back; then a birth covering the
// word takes the maximum, a death covering it keeps the read for its check.
// The lane sets (events' lanes, pending clears) are 64-bit masks in scalar
// registers, combined by scalar ands and ors and used as lane predicates as
// they are; a lone wave issues each event in about 20 instructions.  Groups
// of kUnroll events are read one group ahead through the scalar cache (the
// event buffer has kPad entries past its end, so a read never needs a bound)
// and their checks compared after the group; only a tile's last group masks
// out the events past its end.
__global__ __launch_bounds__(kTBlock) void probe_tiles_kernel(
    const uint64_t* __restrict__ keys, const uint4* __restrict__ packed,
    const int64_t* __restrict__ total_p, int op_bits, uint32_t* slab,
    uint8_t* __restrict__ clob, ProbeFlags* fl) {
    if (fl->skip) return;
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const int64_t n_tiles = fl->n_tiles, total = *total_p;
    const uint64_t top = fl->top;
    for (int64_t tile = (int64_t)blockIdx.x * kTWaves + threadIdx.x / kWave; tile < n_tiles;
         tile += (int64_t)gridDim.x * kTWaves) {
        const int64_t w = (tile << kTileShift) + lane;
        const bool mine = (uint64_t)w < top;
        uint32_t* word = mine ? slab + w : &fl->sink;
        uint32_t v = 0;    // the word's value
        uint64_t clr = 0;  // lanes covered by a death of the current group
        const int64_t e0 = uniform64(wave_find(keys, total, op_bits, (uint64_t)tile, false, lane));
        const int64_t e1 = uniform64(wave_find(keys, total, op_bits, (uint64_t)tile, true, lane));
        auto group = [&](const EventGroup& cur, auto masked, uint32_t live) {
            uint32_t got[kUnroll];
            uint64_t dead[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const uint32_t* e = cur.w + 4 * u;
                uint64_t mask = pair64(e[0], e[1]);
                if constexpr (decltype(masked)::value) mask = ((live >> u) & 1u) ? mask : 0ull;
                const uint32_t s32 = (uint32_t)((int32_t)e[2] >> 31);  // all ones at a group start
                const uint64_t starts = pair64(s32, s32), deaths = pair64(e[3], e[3]);
                v = __builtin_amdgcn_inverse_ballot_w64(clr & starts) ? 0u : v;  // clear
                clr &= ~starts;
                lane_word_store(word, v);
                got[u] = lane_word_load(word);
                v = __builtin_amdgcn_inverse_ballot_w64(mask & ~deaths)
                        ? max(v, e[2] & 0x7FFFFFFFu)
                        : v;
                dead[u] = mask & deaths;
                clr |= dead[u];
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const uint32_t id1 = cur.w[4 * u + 2] & 0x7FFFFFFFu;
                if (__ballot(got[u] != id1) & dead[u]) clob[id1 - 1u] = 1;
            }
        };
        if (e1 > e0) {
            EventGroup cur = group_at(packed, e0);
            int64_t g = e0;
            for (; g + kUnroll <= e1; g += kUnroll) {
                const EventGroup nxt = group_at(packed, g + kUnroll);
                group(cur, std::false_type{}, 0u);
                cur = nxt;
            }
            if (g < e1) group(cur, std::true_type{}, (1u << (uint32_t)(e1 - g)) - 1u);
        }
        v = __builtin_amdgcn_inverse_ballot_w64(clr) ? 0u : v;
        lane_word_store(word, v);
    }
}

__global__ __launch_bounds__(kTBlock) void probe_count_kernel(const uint8_t* __restrict__ clob,
                                                              int64_t n, int64_t* n_clob,
                                                              const ProbeFlags* fl) {
    if (fl->skip) return;
    uint64_t c = 0;
    for (int64_t i = (int64_t)blockIdx.x * kTBlock + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kTBlock)
        c += clob[i];
    c = wave_reduce(c, OpAdd<uint64_t>());
    if ((threadIdx.x & (kWave - 1)) == 0 && c)
        atomicAdd(reinterpret_cast<unsigned long long*>(n_clob), (unsigned long long)c);
}

// Workspace sections.  16- and 8-byte arrays come first, then 4-byte ones,
// with no padding between them, so every extra pair of capacity costs bytes and a
// workspace of probe_workspace_bytes(n, ops, c) holds capacity c exactly.
struct ProbeLayout {
    size_t flags, packed, cnt, partial, keys0, keys1, radix, bstart, dstart, born, dies, big, vals0,
        vals1, end;
};

ProbeLayout probe_layout(int64_t n, int32_t num_ops, int64_t capacity) {
    const size_t nn = (size_t)(n > 0 ? n : 1), ops = (size_t)num_ops + 1;
    const size_t ev = (size_t)(capacity > 0 ? 2 * capacity : 1) + kPad;
    ProbeLayout L;
    size_t at = 0;
    auto take = [&](size_t bytes) {
        const size_t here = at;
        at += bytes;
        return here;
    };
    L.flags = take(256);  // ProbeFlags, padded
    L.packed = take(ev * 16);  // 16-byte events, 16-byte aligned
    L.cnt = take(nn * 8);
    L.partial = take(scan_workspace_bytes((int64_t)nn));
    L.keys0 = take(ev * 8);
    L.keys1 = take(ev * 8);
    L.radix = take(radix_workspace_bytes((int64_t)ev));
    L.bstart = take(ops * 4);
    L.dstart = take(ops * 4);
    L.born = take(nn * 4);
    L.dies = take(nn * 4);
    L.big = take(nn * 4);
    L.vals0 = take(ev * 4);
    L.vals1 = take(ev * 4);
    L.end = at;
    return L;
}

int bit_width(uint64_t x) { return x ? 64 - __builtin_clzll(x) : 0; }

}  // namespace

// capacity: (tensor, tile) pairs the tiled replay can hold; 0 means the
// default of 16 n + 65536.
size_t probe_workspace_bytes(int64_t n, int32_t num_ops, int64_t capacity) {
    if (n < 0 || n >= INT32_MAX || num_ops < 0 || capacity < 0 ||
        capacity > ((int64_t)1 << 40))
        return 0;
    if (capacity == 0) capacity = 16 * n + 65536;
    return probe_layout(n, num_ops, capacity).end;
}

// The largest capacity a workspace of `bytes` holds, or -1 if it is too small
// even for the op-by-op replay.
int64_t probe_capacity(int64_t n, int32_t num_ops, size_t bytes) {
    if (n < 0 || n >= INT32_MAX || num_ops < 0) return -1;
    if (probe_layout(n, num_ops, 0).end > bytes) return -1;
    int64_t lo = 0, hi = (int64_t)1 << 40;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo + 1) / 2;
        if (probe_layout(n, num_ops, mid).end <= bytes) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

hipError_t launch_probe(const int64_t* size, const int32_t* first, const int32_t* last,
                        const int64_t* offset, int64_t n, int32_t num_ops, void* slab,
                        size_t slab_bytes, uint8_t* clob, int64_t* n_clob, void* ws,
                        size_t ws_bytes, int32_t* status, hipStream_t st) {
    const int64_t capacity = probe_capacity(n, num_ops, ws_bytes);
    if (capacity < 0) return hipErrorInvalidValue;
    const ProbeLayout L = probe_layout(n, num_ops, capacity);
    char* w = static_cast<char*>(ws);
    ProbeFlags* fl = reinterpret_cast<ProbeFlags*>(w + L.flags);
    hipLaunchKernelGGL(probe_init_kernel, dim3(1), dim3(1), 0, st, fl, n_clob);
    if (n == 0) return hipGetLastError();

    const int64_t slab_words = (int64_t)(slab_bytes / 4);
    const int64_t max_tiles = (slab_words + 63) >> kTileShift;
    const int op_bits = num_ops > 0 ? bit_width(2 * (uint64_t)num_ops - 1) : 1;
    const int tile_bits = bit_width(max_tiles > 1 ? (uint64_t)(max_tiles - 1) : 0);
    if (op_bits + tile_bits > 64) return hipErrorInvalidValue;
    int64_t* cnt = reinterpret_cast<int64_t*>(w + L.cnt);
    int64_t* partial = reinterpret_cast<int64_t*>(w + L.partial);
    const int64_t* total = partial + (scan_workspace_bytes(n) / sizeof(int64_t) - 1);
    const unsigned nb = (unsigned)((n + kTBlock - 1) / kTBlock);

    hipLaunchKernelGGL(probe_prepare_kernel, dim3(nb), dim3(kTBlock), 0, st, size, first, last,
                       offset, n, num_ops, clob, cnt, fl);
    hipError_t e = device_scan_i64(cnt, n, false, partial, nullptr, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(probe_decide_kernel, dim3(1), dim3(1), 0, st, fl, total, 2 * capacity,
                       slab_words, status);
    if (max_tiles > 0 && capacity > 0) {
        uint64_t* k0 = reinterpret_cast<uint64_t*>(w + L.keys0);
        uint64_t* k1 = reinterpret_cast<uint64_t*>(w + L.keys1);
        uint32_t* v0 = reinterpret_cast<uint32_t*>(w + L.vals0);
        uint32_t* v1 = reinterpret_cast<uint32_t*>(w + L.vals1);
        int32_t* big = reinterpret_cast<int32_t*>(w + L.big);
        hipLaunchKernelGGL(probe_emit_kernel, dim3(nb), dim3(kTBlock), 0, st, size, first, last,
                           offset, n, op_bits, (const int64_t*)cnt, k0, v0, big, fl);
        hipLaunchKernelGGL(probe_emit_big_kernel, dim3((unsigned)min((int64_t)nb, (int64_t)1024)),
                           dim3(kTBlock), 0, st, size, first, last, offset, op_bits,
                           (const int64_t*)cnt, k0, v0, (const int32_t*)big,
                           (const ProbeFlags*)fl);
        bool alt = false;
        e = radix_sort_pairs(k0, v0, k1, v1, 2 * capacity, 0, op_bits + tile_bits, w + L.radix,
                             &alt, st, &fl->skip, total);
        if (e != hipSuccess) return e;
        const uint64_t* ks = alt ? k1 : k0;
        const uint32_t* vs = alt ? v1 : v0;
        uint4* packed = reinterpret_cast<uint4*>(w + L.packed);
        hipLaunchKernelGGL(probe_pack_kernel, dim3((unsigned)min((2 * capacity + kTBlock - 1) / kTBlock,
                                                                 (int64_t)4096)),
                           dim3(kTBlock), 0, st, size, offset, ks, vs, total, op_bits, packed,
                           (const ProbeFlags*)fl);
        const int64_t blocks = min((max_tiles + kTWaves - 1) / kTWaves, (int64_t)1 << 16);
        hipLaunchKernelGGL(probe_tiles_kernel, dim3((unsigned)blocks), dim3(kTBlock), 0, st, ks,
                           (const uint4*)packed, total, op_bits, static_cast<uint32_t*>(slab), clob,
                           fl);
        hipLaunchKernelGGL(probe_count_kernel, dim3((unsigned)min((int64_t)nb, (int64_t)1024)),
                           dim3(kTBlock), 0, st, (const uint8_t*)clob, n, n_clob,
                           (const ProbeFlags*)fl);
    }
    int32_t* b = reinterpret_cast<int32_t*>(w + L.bstart);
    int32_t* d = reinterpret_cast<int32_t*>(w + L.dstart);
    int32_t* born = reinterpret_cast<int32_t*>(w + L.born);
    int32_t* dies = reinterpret_cast<int32_t*>(w + L.dies);
    hipLaunchKernelGGL(probe_ops_kernel, dim3(1), dim3(kPBlock), 0, st, size, first, last, offset,
                       n, num_ops, static_cast<uint32_t*>(slab), slab_words, clob, n_clob, b, d,
                       born, dies, status, (const ProbeFlags*)fl);
    return hipGetLastError();
}

}  // namespace mp
