// Batched greedy-by-size planner: one workgroup per trace, the trace held in LDS.
//
// Method (Section 2.3 greedy_by_size, Section 3.2): tensors are ranked by
// (size desc, first asc, id asc) and each is placed at the lowest offset that
// avoids the byte ranges of the already placed tensors whose lifetimes meet
// its own.  Only lifetime-intersecting pairs interact, so the sequential
// greedy equals evaluating each tensor once all of its "predecessors" --
// intersecting tensors of lower rank -- are placed.  The kernel keeps every
// intersecting pair once in LDS and places tensors in a dataflow schedule
// whose length is the depth of the predecessor DAG, not the tensor count.
//
// Positions q: the trace's tensors ordered by (first, id).  For q < q' the
// pair intersects iff first[q'] <= last[q], so tensor q meets exactly the
// positions (q, reach[q]) to its right, reach[q] = upper_bound(first,
// last[q]), and the positions to its left whose reach passes q (its "left
// list").  For an intersecting pair q < q', q ranks first iff size[q] >=
// size[q'] (equal sizes are ordered by first then id, which is position
// order).
//
// Phases (one workgroup of 512 threads):
//   ingest + checks -> position order -> reach, band lengths, live-bytes
//   deltas, reach histogram -> one prefix pass (band starts, left-list starts,
//   live-bytes maximum) -> left-list fill and predecessor counts -> placement
//   in rounds (a tensor is fitted in the round after its last predecessor)
//   -> outputs.
#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

#ifdef MP_PHASE_TIMING
// Debug builds only: clock stamps of workgroup phases (thread 0), per trace.
constexpr int kPhaseSlots = 8;
__device__ long long g_phase_clock[4096 * kPhaseSlots];
__device__ unsigned int g_dbg[4096 * 8];
#define MP_DBG_MAX(slot, v) \
    do { if (blockIdx.x < 4096) atomicMax(&g_dbg[blockIdx.x * 8 + (slot)], (unsigned)(v)); } while (0)
#define MP_DBG_ADD(slot, v) \
    do { if (blockIdx.x < 4096) atomicAdd(&g_dbg[blockIdx.x * 8 + (slot)], (unsigned)(v)); } while (0)
#define MP_STAMP(slot)                                                              \
    do {                                                                            \
        if (threadIdx.x == 0 && blockIdx.x < 4096)                                  \
            g_phase_clock[blockIdx.x * kPhaseSlots + (slot)] = clock64();           \
    } while (0)
#else
#define MP_STAMP(slot) do { } while (0)
#define MP_DBG_MAX(slot, v) do { } while (0)
#define MP_DBG_ADD(slot, v) do { } while (0)
#endif

namespace {

constexpr int kBatchBlock = 512;
constexpr uint32_t kSmallK = 16;           // neighbours of a tensor fitted by a lane quad
constexpr uint32_t kMidK = 64;             // ... by a 16-lane row; more: by the whole wave
constexpr int kSlots = 4;                  // neighbours per lane in quads, rows and waves
constexpr uint32_t kCoopChunk = 64u * kSlots;
constexpr uint32_t kBigClass = 0x80000000u;  // pending-count flag: more than kSmallK neighbours
constexpr uint32_t kCountMask = 0x7FFFFFFFu;

// A tensor's LDS word: offset (units) in the high half, size (units) in the
// low half; the offset half is kUnplaced until the tensor is placed.  An
// unplaced word never overlaps a candidate range: offsets stay below
// 0xFFFFFFFF because the sizes of a trace sum to at most 0xFFFFFFFE units.
__device__ __forceinline__ uint32_t word_off(uint64_t w) { return (uint32_t)(w >> 32); }
__device__ __forceinline__ uint32_t word_end(uint64_t w) {
    return (uint32_t)(w >> 32) + (uint32_t)w;
}

// Neighbour q' of q ranks after q (a successor) iff it is smaller, or equal
// in size and later in position order.
__device__ __forceinline__ bool ranks_after(uint32_t s_other, uint32_t id_other, uint32_t s,
                                            uint32_t q) {
    return (s_other < s) | ((s_other == s) & (id_other > q));
}

// Maximum over the 64 lanes, returned to every lane: DPP row shifts build
// row-wise prefix maxima, row broadcasts carry them across rows, lane 63
// ends up with the total.  All 64 lanes must be active.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false));
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Maximum over each quad of lanes (4g .. 4g+3), returned to all four:
// quad permutations swap lanes 1 apart, then 2 apart.
__device__ __forceinline__ uint32_t quad_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
    return v;
}
// Maximum over each row of 16 lanes, returned to all of them: rotations by
// 8, 4, 2 and 1 within the row.
__device__ __forceinline__ uint32_t row_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x124, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x122, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x121, 0xF, 0xF, false));
    return v;
}
// Lane 0 of each quad / of each row, to every lane of it.
__device__ __forceinline__ uint32_t quad_first(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x00, 0xF, 0xF, false);
}
__device__ __forceinline__ uint32_t row_first(uint32_t v, int lane) {
    const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
    const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
    const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
    const uint32_t r3 = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
    return lane < 32 ? (lane < 16 ? r0 : r1) : (lane < 48 ? r2 : r3);
}

template <int BLOCK>
__device__ void bitonic_sort_u64(uint64_t* keys, int m) {
    for (int k = 2; k <= m; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < (m >> 1); i += BLOCK) {
                // i-th compare-exchange pair of this stage
                const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1));
                const int hi = lo | j;
                const uint64_t a = keys[lo], b = keys[hi];
                const bool up = (lo & k) == 0;
                if ((a > b) == up) {
                    keys[lo] = b;
                    keys[hi] = a;
                }
            }
            __syncthreads();
        }
    }
}

// Neighbour k of tensor q in its neighbour sequence: the left list first
// (k < L), then the right band q + 1 .. q + R.  `lv` is the left-list entry
// lst[lb + k] (ignored for k >= L).  Slots past the end (k >= K) map to q
// itself, which is unplaced and never a successor of itself.
__device__ __forceinline__ uint32_t neighbour(uint32_t k, uint32_t L, uint32_t K, uint32_t q,
                                              uint32_t lv) {
    return k < L ? lv : (k < K ? q + 1 + (k - L) : q);
}

// Ready lists, one per class (at most kSmallK neighbours, or more).  Each
// tensor is appended once; the tensors released during a round go after
// `end` (the end of the round's own range), counted by `cnt`.
struct ReadyLists {
    uint16_t* slot[2];
    uint32_t end[2];
    uint32_t* cnt[2];
};

// Exclusive prefix over the wave's lanes of a small count v (< 8), and the
// wave total: one ballot per bit.  All 64 lanes must be active.
__device__ __forceinline__ uint32_t wave_prefix_small(uint32_t v, uint32_t& total) {
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int bit = 0; bit < 3; ++bit) {
        const uint64_t m = __ballot((v >> bit) & 1u);
        const uint32_t below = __builtin_amdgcn_mbcnt_hi(
            (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        pre += below << bit;
        tot += (uint32_t)__popcll(m) << bit;
    }
    total = tot;
    return pre;
}

// Decrement the pending counts of the successors among M (<= 7) gathered
// neighbours (dec[j] is 1 for a successor, else 0: the atomics then issue
// back to back) and append those that reach zero to their class list, one
// list reservation per wave.  All 64 lanes must be active.
template <int M>
__device__ __forceinline__ void release_successors(const uint32_t (&dec)[M],
                                                   const uint32_t (&ids)[M], uint32_t* rem,
                                                   const ReadyLists& rl, int lane) {
    static_assert(M < 8, "counts must fit three bits");
    uint32_t old[M];
#pragma unroll
    for (int j = 0; j < M; ++j) old[j] = atomicSub(rem + ids[j], dec[j]);
    uint32_t ready[2] = {0, 0};
#pragma unroll
    for (int j = 0; j < M; ++j) {
        const bool r = dec[j] && (old[j] & kCountMask) == 1u;
        ready[0] |= (r && !(old[j] & kBigClass) ? 1u : 0u) << j;
        ready[1] |= (r && (old[j] & kBigClass) ? 1u : 0u) << j;
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        if (!__ballot(ready[c] != 0)) continue;
        uint32_t total;
        const uint32_t pre = wave_prefix_small((uint32_t)__popc(ready[c]), total);
        uint32_t base = 0;
        if (lane == 0) base = atomicAdd(rl.cnt[c], total);
        uint32_t at = rl.end[c] + (uint32_t)__builtin_amdgcn_readlane((int)base, 0) + pre;
#pragma unroll
        for (int j = 0; j < M; ++j)
            if (ready[c] >> j & 1u) rl.slot[c][at++] = (uint16_t)ids[j];
    }
}

// Whole-wave placement of tensor q (all 64 lanes active, arguments uniform):
// the neighbour sequence is swept in chunks of 256, each lane holding up to 4
// neighbours; within a chunk the candidate offset jumps to the highest end
// overlapping [x, x + s) until nothing in the chunk overlaps, and chunks are
// revisited until a full lap leaves x alone.  Then q is published and its
// successors' pending counts are decremented.
__device__ void place_wave(uint32_t q, uint32_t s, uint32_t lb, uint32_t L, uint32_t K,
                           uint64_t* ofsz, const uint16_t* lst, uint32_t* rem,
                           const ReadyLists& rl, int lane) {
    const uint32_t nch = (K + kCoopChunk - 1) / kCoopChunk;
    uint32_t id[kSlots], co[kSlots], ce[kSlots], cs[kSlots];
    auto load = [&](uint32_t kb) {
        uint32_t lv[kSlots];
#pragma unroll
        for (int r = 0; r < kSlots; ++r) {
            const uint32_t k = kb + r * kWave + lane;
            lv[r] = lst[k < L ? lb + k : lb];  // in bounds: the list area is padded
        }
        uint64_t w[kSlots];
#pragma unroll
        for (int r = 0; r < kSlots; ++r) {
            id[r] = neighbour(kb + r * kWave + lane, L, K, q, lv[r]);
            w[r] = ofsz[id[r]];
        }
#pragma unroll
        for (int r = 0; r < kSlots; ++r) {
            co[r] = word_off(w[r]);
            ce[r] = word_end(w[r]);
            cs[r] = (uint32_t)w[r];
        }
    };
    uint32_t x = 0, clean = 0, c = 0;
    while (clean < nch) {
        load(c * kCoopChunk);
        bool moved = false;
        while (true) {  // jump past the highest end overlapping [x, x + s)
            bool ov = false;
            uint32_t mx = 0;
#pragma unroll
            for (int r = 0; r < kSlots; ++r) {
                if (co[r] < x + s && x < ce[r]) {
                    ov = true;
                    mx = max(mx, ce[r]);
                }
            }
            if (!__ballot(ov)) break;
            x = wave_max_u32(mx);
            moved = true;
        }
        clean = moved ? 1u : clean + 1u;
        c = (c + 1 == nch) ? 0u : c + 1;
    }
    if (lane == 0) ofsz[q] = ((uint64_t)x << 32) | s;
    for (uint32_t cc = 0; cc < nch; ++cc) {
        if (nch > 1) load(cc * kCoopChunk);
        uint32_t dec[kSlots];
#pragma unroll
        for (int r = 0; r < kSlots; ++r) {
            const uint32_t k = cc * kCoopChunk + r * kWave + lane;
            dec[r] = ((k < K) & ranks_after(cs[r], id[r], s, q)) ? 1u : 0u;
        }
        release_successors(dec, id, rem, rl, lane);
    }
}

// A tensor being fitted by a lane group: its id, size, left-list start, left
// length and neighbour count (all lanes of the group hold the same values).
struct Item {
    uint32_t q, s, lb, L, K;
};

__device__ __forceinline__ Item load_item(uint32_t q, bool has, const uint64_t* ofsz,
                                          const uint16_t* lbeg, const uint16_t* reach) {
    Item it{0, 0, 0, 0, 0};
    if (has) {
        it.q = q;
        it.s = (uint32_t)ofsz[q];
        it.lb = lbeg[q];
        it.L = (uint32_t)lbeg[q + 1] - it.lb;
        it.K = it.L + (uint32_t)reach[q] - q - 1;
    }
    return it;
}

// The neighbours k = g + G * r (r < kSlots) of a group's tensor, for the
// lane at position g of a group of G lanes: ids, ranges [o, e) (o = kUnplaced
// for an unplaced or missing neighbour, which never overlaps) and sizes.
// `live` is false for groups without a tensor.
template <int G>
__device__ __forceinline__ void gather_group(const Item& it, bool live, uint32_t g,
                                             const uint64_t* ofsz, const uint16_t* lst,
                                             uint32_t (&id)[kSlots], uint32_t (&o)[kSlots],
                                             uint32_t (&e)[kSlots], uint32_t (&z)[kSlots]) {
    uint32_t lv[kSlots];
#pragma unroll
    for (int r = 0; r < kSlots; ++r) {
        const uint32_t k = g + G * r;
        lv[r] = lst[k < it.L ? it.lb + k : it.lb];  // in bounds: the list area is padded
    }
    uint64_t w[kSlots];
#pragma unroll
    for (int r = 0; r < kSlots; ++r) {
        const uint32_t k = g + G * r;
        id[r] = live ? neighbour(k, it.L, it.K, it.q, lv[r]) : 0u;
        w[r] = ofsz[id[r]];
    }
#pragma unroll
    for (int r = 0; r < kSlots; ++r) {
        const bool in = live && (g + G * r) < it.K;
        o[r] = in ? word_off(w[r]) : kUnplaced;
        e[r] = word_end(w[r]);
        z[r] = (uint32_t)w[r];
    }
}

// Highest end among the lane's ranges that overlap [x, x + s), 0 if none.
__device__ __forceinline__ uint32_t overlap_end(const uint32_t (&o)[kSlots],
                                                const uint32_t (&e)[kSlots], uint32_t x,
                                                uint32_t s) {
    uint32_t m = 0;
#pragma unroll
    for (int r = 0; r < kSlots; ++r) m = (o[r] < x + s && x < e[r]) ? max(m, e[r]) : m;
    return m;
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
    __shared__ uint32_t nready[2][3];  // per class: tensors appended in rounds r % 3

    // LDS layout (N = cap_n tensor slots, P = cap_pairs list slots):
    //   A [8N]     first[N] (i32)                  -> placement words ofsz[N]
    //   B [4N+4]   band lengths -> band starts     -> ready queue (u16)
    //   C [4N+4]   live-bytes deltas -> left-list fill cursors
    //   D [4N+4]   reach histogram -> pending predecessor counts
    //   E [2N+2]   left-list starts (u16)
    //   F [2N]     reach (u16)
    //   G [2P+32]  left lists (u16 positions; padded for unconditional reads)
    //   D..G hold the u64 sort keys of an unsorted trace before the reach pass.
    const size_t N = (size_t)cap_n;
    int32_t* fst = reinterpret_cast<int32_t*>(smem);
    uint64_t* ofsz = reinterpret_cast<uint64_t*>(smem);
    const uint32_t* szw = reinterpret_cast<const uint32_t*>(smem);  // size half at 2q
    uint32_t* band = reinterpret_cast<uint32_t*>(smem + 8 * N);
    uint16_t* readyq = reinterpret_cast<uint16_t*>(smem + 8 * N);
    uint32_t* live = reinterpret_cast<uint32_t*>(smem + 12 * N + 4);
    uint32_t* cursor = live;
    uint32_t* hist = reinterpret_cast<uint32_t*>(smem + 16 * N + 8);
    uint32_t* rem = hist;
    uint64_t* keys = reinterpret_cast<uint64_t*>(smem + 16 * N + 8);
    uint16_t* lbeg = reinterpret_cast<uint16_t*>(smem + 20 * N + 12);
    uint16_t* reach = reinterpret_cast<uint16_t*>(smem + 22 * N + 14);
    uint16_t* lst = reinterpret_cast<uint16_t*>(smem + 24 * N + 14);
    uint32_t* scratch = reinterpret_cast<uint32_t*>(red);

    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    MP_STAMP(0);
    if (tid == 0) {
        nready[0][0] = nready[0][1] = nready[0][2] = 0;
        nready[1][0] = nready[1][1] = nready[1][2] = 0;
    }
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
    flags = block_reduce<BLOCK>(flags, OpOr<uint32_t>(), scratch);
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
    MP_STAMP(1);
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
    int m = 1;
    while (m < n) m <<= 1;
    if (flags & 2u) {
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
    uint32_t su_r[ITEMS];
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        su_r[k] = 0;
        if (q < n) {
            su_r[k] = (uint32_t)((uint64_t)s_r[k] >> sh);
            fst[q] = f_r[k];
        }
    }
    for (int i = tid; i <= n; i += BLOCK) {
        live[i] = 0;
        hist[i] = 0;
    }
    __syncthreads();
    MP_STAMP(2);

    // ---- reach (galloping search), band lengths, live-bytes deltas, reach histogram
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        if (q < n) {
            const int32_t l = l_r[k];
            int known = q, step = 1, probe = q + 1;  // first[known] <= l
            while (probe < n && fst[probe] <= l) {
                known = probe;
                step <<= 1;
                probe = q + step;
            }
            int a = known + 1, z = probe < n ? probe : n;
            while (a < z) {
                const int mid = (a + z) >> 1;
                if (fst[mid] <= l) a = mid + 1;
                else z = mid;
            }
            reach[q] = (uint16_t)a;
            band[q] = (uint32_t)(a - q - 1);
            atomicAdd(&live[q], su_r[k]);
            atomicAdd(&live[a], 0u - su_r[k]);
            atomicAdd(&hist[a], 1u);
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {  // first[] is no longer needed
        const int q = tid + k * BLOCK;
        if (q < n) ofsz[q] = ((uint64_t)kUnplaced << 32) | su_r[k];
    }
    MP_STAMP(3);

    // ---- one prefix pass over positions j (contiguous chunk per thread):
    //   band start      = sum of band lengths before j        (pair index base)
    //   left-list start = sum over i < j of #{q : q < i < reach[q]}
    //                   = j(j-1)/2 - j * H(<j) + sum_{r<j} r * hist[r],
    //     since position i has i - #{q : reach[q] <= i} left neighbours;
    //   live bytes      = running sum of the deltas (its maximum is the bound).
    // The three integer sums share one 64-bit word: band (24 bits, at most
    // n(n-1)/2), hist count (13 bits, at most n) and r * hist (25 bits).
    uint32_t live_max;
    uint32_t n_pairs;
    {
        const int chunk = (n + BLOCK - 1) / BLOCK;
        const int a0 = min(n, tid * chunk), a1 = min(n, a0 + chunk);
        auto pack = [](uint32_t bl, uint32_t h, uint32_t j) {
            return ((uint64_t)bl << 38) | ((uint64_t)h << 25) | (uint64_t)(h * j);
        };
        uint64_t ps = 0;
        uint32_t ds = 0;
        for (int i = a0; i < a1; ++i) {
            ps += pack(band[i], hist[i], (uint32_t)i);
            ds += live[i];
        }
        uint64_t ptot;
        uint64_t prun = block_exclusive_sum<BLOCK>(ps, &ptot, red);
        uint32_t dtot;
        uint32_t drun = block_exclusive_sum<BLOCK>(ds, &dtot, scratch);
        uint32_t lm = 0;
        for (int i = a0; i < a1; ++i) {
            const uint32_t bl = band[i], h = hist[i], dl = live[i];
            const uint32_t hb = (uint32_t)(prun >> 25) & 0x1FFFu;
            const uint32_t rh = (uint32_t)prun & 0x1FFFFFFu;
            const uint32_t ls = (uint32_t)(i * (i - 1) / 2) - (uint32_t)i * hb + rh;
            band[i] = (uint32_t)(prun >> 38);
            lbeg[i] = (uint16_t)ls;
            cursor[i] = ls;
            rem[i] = 0;
            drun += dl;
            lm = lm > drun ? lm : drun;
            prun += pack(bl, h, (uint32_t)i);
        }
        n_pairs = (uint32_t)(ptot >> 38);
        if (tid == 0) {
            band[n] = n_pairs;
            lbeg[n] = (uint16_t)n_pairs;
        }
        live_max = block_reduce<BLOCK>(lm, OpMax<uint32_t>(), scratch);
    }
    if (n_pairs > (uint32_t)cap_pairs) {
        if (tid == 0) raise_status(status, MP_ENOSPC);
        return;
    }
    MP_STAMP(4);

    // ---- left lists and pending predecessor counts, balanced over the pairs:
    // pair index p -> (q, j), j = q + 1 + (p - band start of q)
    {
        const uint32_t per = (n_pairs + BLOCK - 1) / BLOCK;
        const uint32_t p_lo = min(n_pairs, (uint32_t)tid * per), p_hi = min(n_pairs, p_lo + per);
        if (p_lo < p_hi) {
            int a = 0, z = n;  // last position whose band starts at or before p_lo
            while (a < z) {
                const int mid = (a + z + 1) >> 1;
                if (band[mid] <= p_lo) a = mid;
                else z = mid - 1;
            }
            int q = a;
            uint32_t base = band[q], nxt = band[q + 1];
            uint32_t sq = szw[2 * q];
            for (uint32_t p = p_lo; p < p_hi; ++p) {
                while (nxt <= p) {
                    ++q;
                    base = nxt;
                    nxt = band[q + 1];
                    sq = szw[2 * q];
                }
                const uint32_t j = (uint32_t)q + 1 + (p - base);
                lst[atomicAdd(&cursor[j], 1u)] = (uint16_t)q;
                atomicAdd(&rem[sq >= szw[2 * j] ? j : (uint32_t)q], 1u);
            }
        }
    }
    __syncthreads();

    // ---- ready lists: tensors with more than kSmallK neighbours form the
    // big class (flag in the pending count); tensors without predecessors
    // seed the lists
    {
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int q = tid + k * BLOCK;
            if (q < n) {
                const uint32_t K = (uint32_t)lbeg[q + 1] - lbeg[q] + (uint32_t)reach[q] - q - 1;
                const uint32_t r = rem[q] | (K > kSmallK ? kBigClass : 0u);
                rem[q] = r;
                if ((r & kCountMask) == 0) {
                    const int c = (r & kBigClass) ? 1 : 0;
                    readyq[c * N + atomicAdd(&nready[c][2], 1u)] = (uint16_t)q;
                }
            }
        }
    }
    __syncthreads();
    MP_STAMP(5);

    // ---- placement in rounds (Kahn's order over the predecessor DAG): round
    // r fits every tensor released in round r - 1 -- all of its predecessors
    // are placed, and no two of them intersect -- with one lane quad per
    // small-class tensor (four neighbours per lane) and one 16-lane row per
    // big-class tensor (the whole wave past kMidK neighbours), packed into as
    // few waves as possible.  A group gathers the neighbours' words (the
    // placed ones are exactly the predecessors), moves the candidate offset
    // past the highest overlapping end until nothing overlaps, publishes the
    // word and decrements the successors' pending counts; those reaching zero
    // are appended for the next round.  Per-round append counters rotate over
    // three slots so that one barrier per round suffices.
    {
        const int lane = tid & (kWave - 1);
        const uint32_t g4 = lane & 3, g16 = lane & 15;
        const uint32_t quad = (uint32_t)tid >> 2, row = (uint32_t)tid >> 4;
        constexpr uint32_t kQuads = BLOCK / 4, kRows = BLOCK / 16;
        uint32_t b0 = 0, e0 = nready[0][2], b1 = 0, e1 = nready[1][2];
        for (int round = 0; b0 < e0 || b1 < e1; ++round) {
            if (round > n) {  // cannot happen: every round places a tensor
                if (tid == 0) raise_status(status, MP_EDEVICE);
                break;
            }
            const int cur = round % 3, nxt = (round + 1) % 3;
            if (tid == 0) nready[0][nxt] = nready[1][nxt] = 0;
            const ReadyLists rl{{readyq, readyq + N}, {e0, e1}, {&nready[0][cur], &nready[1][cur]}};
#ifdef MP_PHASE_TIMING
            if (tid == 0) MP_DBG_ADD(0, 1u);
#endif
            for (uint32_t it = 0;; ++it) {
                // small tensors fill quads from the first wave up, big ones
                // rows from the last wave down
                const uint32_t i0 = b0 + quad + kQuads * it;
                const uint32_t i1 = b1 + (kRows - 1 - row) + kRows * it;
                const bool hs = i0 < e0, hb = i1 < e1;
                const bool any_s = __ballot(hs) != 0, any_b = __ballot(hb) != 0;
                if (!any_s && !any_b) break;
#ifdef MP_PHASE_TIMING
                if (lane == 0) MP_DBG_ADD(1, 1u);
#endif
                if (any_s) {
                    const Item is = load_item(hs ? readyq[i0] : 0u, hs, ofsz, lbeg, reach);
                    uint32_t id[kSlots], o[kSlots], e[kSlots], z[kSlots];
                    gather_group<4>(is, hs, g4, ofsz, lst, id, o, e, z);
                    uint32_t x = 0;
                    while (true) {  // jump past the highest overlapping end until none moves
                        const uint32_t m = quad_max_u32(overlap_end(o, e, x, is.s));
                        const bool mv = m > x;
                        x = mv ? m : x;
#ifdef MP_PHASE_TIMING
                        if (lane == 0) MP_DBG_ADD(2, 1u);
#endif
                        if (!__ballot(mv)) break;
                    }
                    if (hs && g4 == 0) ofsz[is.q] = ((uint64_t)x << 32) | is.s;
                    uint32_t dec[kSlots];
#pragma unroll
                    for (int r = 0; r < kSlots; ++r)
                        dec[r] = (hs & ((g4 + 4 * r) < is.K) & ranks_after(z[r], id[r], is.s, is.q))
                                     ? 1u : 0u;
                    release_successors(dec, id, rem, rl, lane);
                }
                if (any_b) {
                    const Item ib = load_item(hb ? readyq[N + i1] : 0u, hb, ofsz, lbeg, reach);
                    const bool mid = hb && ib.K <= kMidK;
                    uint32_t id[kSlots], o[kSlots], e[kSlots], z[kSlots];
                    gather_group<16>(ib, mid, g16, ofsz, lst, id, o, e, z);
                    uint32_t x = 0;
                    while (true) {
                        const uint32_t m = row_max_u32(overlap_end(o, e, x, ib.s));
                        const bool mv = m > x;
                        x = mv ? m : x;
#ifdef MP_PHASE_TIMING
                        if (lane == 0) MP_DBG_ADD(3, 1u);
#endif
                        if (!__ballot(mv)) break;
                    }
                    if (mid && g16 == 0) ofsz[ib.q] = ((uint64_t)x << 32) | ib.s;
                    uint32_t dec[kSlots];
#pragma unroll
                    for (int r = 0; r < kSlots; ++r)
                        dec[r] = (mid & ((g16 + 16 * r) < ib.K) & ranks_after(z[r], id[r], ib.s, ib.q))
                                     ? 1u : 0u;
                    release_successors(dec, id, rem, rl, lane);
                    uint64_t wide = __ballot(hb && !mid && g16 == 0);
                    while (wide) {
                        const int src = __ffsll((long long)wide) - 1;
                        wide &= wide - 1;
                        place_wave((uint32_t)__builtin_amdgcn_readlane((int)ib.q, src),
                                   (uint32_t)__builtin_amdgcn_readlane((int)ib.s, src),
                                   (uint32_t)__builtin_amdgcn_readlane((int)ib.lb, src),
                                   (uint32_t)__builtin_amdgcn_readlane((int)ib.L, src),
                                   (uint32_t)__builtin_amdgcn_readlane((int)ib.K, src), ofsz,
                                   lst, rem, rl, lane);
                    }
                }
            }
            __syncthreads();
            b0 = e0;
            e0 += nready[0][cur];
            b1 = e1;
            e1 += nready[1][cur];
        }
    }
    __syncthreads();
    MP_STAMP(6);

    // ---- outputs
    uint32_t pk = 0;
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        if (q < n) {
            const uint64_t w = ofsz[q];
            offset_out[lo + id_r[k]] = (int64_t)((uint64_t)word_off(w) << sh);
            const uint32_t e = word_end(w);
            pk = pk > e ? pk : e;
        }
    }
    pk = block_reduce<BLOCK>(pk, OpMax<uint32_t>(), scratch);
    if (tid == 0) {
        peak_out[b] = (int64_t)((uint64_t)pk << sh);
        if (lb_out) lb_out[b] = (int64_t)((uint64_t)live_max << sh);
    }
    MP_STAMP(7);
}

__global__ void reset_status_kernel(int32_t* status) { *status = MP_OK; }

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

#ifdef MP_PHASE_TIMING
extern "C" int32_t mp_debug_counters(unsigned* host_out, int64_t n, int reset) {
    if (n > 4096 * 8) n = 4096 * 8;
    if (reset) {
        static unsigned zeros[4096 * 8];
        return hipMemcpyToSymbol(HIP_SYMBOL(g_dbg), zeros, sizeof(zeros)) == hipSuccess ? MP_OK : MP_EDEVICE;
    }
    return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_dbg), n * sizeof(unsigned), 0,
                               hipMemcpyDeviceToHost) == hipSuccess ? MP_OK : MP_EDEVICE;
}
extern "C" int32_t mp_debug_phase_clock(long long* host_out, int64_t n) {
    if (n > 4096 * kPhaseSlots) n = 4096 * kPhaseSlots;
    return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_phase_clock), n * sizeof(long long), 0,
                               hipMemcpyDeviceToHost) == hipSuccess
               ? MP_OK
               : MP_EDEVICE;
}
#endif

hipError_t launch_reset_status(int32_t* status, hipStream_t st) {
    hipLaunchKernelGGL(reset_status_kernel, dim3(1), dim3(1), 0, st, status);
    return hipGetLastError();
}

// LDS bytes per workgroup: 24 per tensor slot + 16, plus 2 per pair slot + 32.
// Traces up to about 2000 tensors get a budget that lets two workgroups share
// a CU's 160 KiB of LDS.  Pair slots stay below 2^16 (left-list starts are
// u16), which both budgets imply.  The sort keys (8 bytes per power-of-two
// slot) must fit from region D on.
BatchShape batch_shape(int64_t max_trace_len) {
    BatchShape s{};
    if (max_trace_len < 0 || max_trace_len > MP_BATCH_MAX_TRACE_LEN) return s;
    const int64_t cap_n = max_trace_len < 1 ? 1 : max_trace_len;
    const int64_t fixed = 24 * cap_n + 16;
    const int64_t budget = (fixed <= 48 * 1024) ? 78 * 1024 : 156 * 1024;
    int64_t pairs = (budget - fixed - 32) / 2;
    pairs &= ~(int64_t)7;
    if (pairs > 65528) pairs = 65528;
    int64_t m = 1;
    while (m < cap_n) m <<= 1;
    if (8 * cap_n + 2 * pairs + 40 < 8 * m) return s;  // keys would not fit (never for <= 4096)
    s.cap_n = (int32_t)cap_n;
    s.cap_pairs = (int32_t)pairs;
    s.lds_bytes = (size_t)(fixed + 2 * pairs + 32);
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
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mp
