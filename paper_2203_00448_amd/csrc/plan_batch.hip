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
// list", stored as one byte per entry: the distance back, or the slot of one
// of a few long-lived tensors).  For an intersecting pair q < q', q ranks
// first iff size[q] >= size[q'] (equal sizes are ordered by first then id,
// which is position order).
//
// Phases (one workgroup of 512 threads):
//   ingest + checks -> position order -> reach, band lengths, live-bytes
//   deltas, reach histogram, long tensors -> one prefix pass (band starts,
//   left-list starts, live-bytes maximum, largest neighbour count) ->
//   left-list fill and predecessor counts -> placement words -> placement in
//   rounds (a tensor is fitted in the round after its last predecessor) ->
//   outputs.
// A trace the LDS path cannot hold -- sizes summing to 2^31 units or more,
// more intersecting pairs than the LDS list capacity, more than 32 long
// tensors, or under BEST_FIT a tensor meeting more than 256 others -- is
// planned by the same workgroup on the general path (plan_general): the
// greedy taken literally, one tensor at a time in rank order, 64-bit offsets,
// its working lists in the workspace.  No valid trace is refused.
#include <type_traits>

#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

#ifdef MP_PHASE_TIMING
// Debug builds only: clock stamps of workgroup phases (thread 0), per trace.
constexpr int kPhaseSlots = 8;
__device__ long long g_phase_clock[4096 * kPhaseSlots];
__device__ unsigned int g_dbg[4096 * 8];
#define MP_DBG_ADD(slot, v) \
    do { if (blockIdx.x < 4096) atomicAdd(&g_dbg[blockIdx.x * 8 + (slot)], (unsigned)(v)); } while (0)
#define MP_STAMP(slot)                                                              \
    do {                                                                            \
        if (threadIdx.x == 0 && blockIdx.x < 4096)                                  \
            g_phase_clock[blockIdx.x * kPhaseSlots + (slot)] = clock64();           \
    } while (0)
#else
#define MP_STAMP(slot) do { } while (0)
#define MP_DBG_ADD(slot, v) do { } while (0)
#endif

namespace {

// Threads per trace: 256 up to 2048 tensors (four workgroups a CU then have
// four waves a SIMD, 128 VGPRs each, and measured faster than 512 threads
// with 64), 512 for longer traces (at most eight tensor slots a thread).
constexpr int kBatchBlock = 256;
constexpr int kBatchBlockLong = 512;
constexpr int kMaxItems = 8;
// Issue priority by pace.  Four traces share a CU and the kernel lasts as
// long as the slowest; the wave arbiter favours the oldest waves, so the
// workgroup dispatched last to a CU was the slowest.  Each round a trace
// compares its progress with a nominal pace (kPaceSetup ticks of the 100 MHz
// clock from its workgroup's start -- all of a batch's workgroups start
// together when they fit the device at once -- then kPaceRound a round:
// about the averages of 2000-tensor traces four to a CU) and issues with
// priority min(rounds behind, 3).  Where every trace is behind, or none, all keep the same
// priority, as without it.  2000-tensor batch: 143 -> 132 us.
constexpr int64_t kPaceSetup = 3400;
constexpr int64_t kPaceRound = 350;
constexpr int kLaneSlots = 8;                   // neighbours a lane holds while fitting
constexpr int kBestSlots = 4;                   // ... in the whole-wave BEST_FIT sort
constexpr uint32_t kCoopChunk = (uint32_t)kWave * kLaneSlots;
constexpr uint32_t kBestMaxK = (uint32_t)kWave * kBestSlots;  // BEST_FIT on the LDS path

// Ready classes by neighbour count K: the lanes a tensor is fitted by.
// 0: K <= 8, one lane; 1: K <= 16, two; 2: K <= 32, four; 3: K <= 64,
// eight; 4: more, the whole wave (under BEST_FIT every K > 8).
constexpr int kClasses = 5;
constexpr int kWideClass = 4;

// A tensor's LDS placement word: size (units) in the low half; the high half
// is the offset (units, below 2^31) once placed, and before that bit 31 set,
// the tensor's count in its ready class's 4-bit field (1 << (12 + 4 c)) and
// the number of unplaced predecessors in bits 0-11 (a trace has at most 4096
// tensors).  An unplaced word never overlaps a candidate range: every
// candidate end plus the size being fitted stays below 2^31 units, because
// the trace's sizes sum to less (the greedy's peak never exceeds that sum).
constexpr uint32_t kUnplacedBit = 0x80000000u;
constexpr uint32_t kClassShift = 12;
constexpr uint32_t kPendMask = (1u << kClassShift) - 1;
__device__ __forceinline__ uint32_t class_bits(uint32_t c) { return 1u << (kClassShift + 4u * c); }
constexpr uint64_t kFastMaxUnits = 0x7FFFFFFFull;
// A slot past the tensor's neighbour count: sorts after every range, never
// overlaps one and names no successor.
constexpr uint32_t kNoSlot = 0xFFFFFFFFu;

// Left-list entries (one byte): 1 .. kMaxDist is the distance back to the
// neighbour's position; kLongBase + s names long tensor s (a tensor whose
// band reaches further than kMaxDist), whose position is in a small table.
constexpr uint32_t kLongSlots = 32;
constexpr uint32_t kLongBase = 256 - kLongSlots;
constexpr uint32_t kMaxDist = kLongBase - 1;

__device__ __forceinline__ uint32_t ready_class(uint32_t K, bool best) {
    if (K <= 8) return 0u;
    if (best) return (uint32_t)kWideClass;
    return K <= 16 ? 1u : (K <= 32 ? 2u : (K <= 64 ? 3u : (uint32_t)kWideClass));
}

__device__ __forceinline__ uint32_t word_off(uint64_t w) { return (uint32_t)(w >> 32); }
__device__ __forceinline__ uint32_t word_end(uint64_t w) {
    return (uint32_t)(w >> 32) + (uint32_t)w;
}

// 16-bit counters packed two per 32-bit LDS word (entry i in half i & 1;
// LDS atomics are 32-bit).  No entry ever leaves [0, 2^16), so a carry or
// borrow never reaches the neighbouring half.
__device__ __forceinline__ uint32_t half_shift(uint32_t i) { return (i & 1u) << 4; }
__device__ __forceinline__ uint32_t packed_get(const uint32_t* w, uint32_t i) {
    return (w[i >> 1] >> half_shift(i)) & 0xFFFFu;
}
__device__ __forceinline__ uint32_t packed_add(uint32_t* w, uint32_t i, uint32_t v) {
    return (atomicAdd(w + (i >> 1), v << half_shift(i)) >> half_shift(i)) & 0xFFFFu;
}

// The trace's left lists and long-tensor table, as the placement reads them.
struct LeftLists {
    const uint8_t* ent;       // entries, tensor q's at [lbeg[q], lbeg[q + 1])
    const uint16_t* longtab;  // positions of the long tensors
};

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

// Maximum over each aligned group of G lanes (G a power of two up to 64,
// per lane; the lanes of a group agree on it), returned to the group: swaps
// within pairs and quads (quad_perm), between the quads of each half row
// (half-row mirror) and the halves of each row (rotation by 8); groups of
// 32 and 64 lanes combine the row maxima read from the first lane of each
// row.  All 64 lanes must be active.
__device__ __forceinline__ uint32_t group_max_u32(uint32_t v, uint32_t G) {
    uint32_t t = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
    v = G >= 2 ? t : v;
    t = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
    v = G >= 4 ? t : v;
    t = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
    v = G >= 8 ? t : v;
    t = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false));
    v = G >= 16 ? t : v;
    if (__ballot(G >= 32u)) {
        const uint32_t m0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
        const uint32_t m1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
        const uint32_t m2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
        const uint32_t m3 = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
        const uint32_t h0 = max(m0, m1), h1 = max(m2, m3);
        const uint32_t h = (threadIdx.x & 32u) ? h1 : h0;
        v = G >= 64 ? max(h0, h1) : (G >= 32 ? h : v);
    }
    return v;
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

// Inclusive sum over the 64 lanes (DPP row shifts, then row broadcasts).
// All 64 lanes must be active.
__device__ __forceinline__ uint32_t wave_inclusive_sum_dpp(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);
    return v;
}

// Inclusive sum of 64-bit values over the 64 lanes (both halves moved by DPP
// from the same source lane, added in 64 bits).  All 64 lanes must be active.
__device__ __forceinline__ uint64_t wave_inclusive_sum64_dpp(uint64_t v) {
#define MP_STEP64(ctrl, rows)                                                                   \
    {                                                                                           \
        const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, ctrl,    \
                                                                  rows, 0xF, false);           \
        const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), \
                                                                  ctrl, rows, 0xF, false);     \
        v += ((uint64_t)hi << 32) | lo;                                                         \
    }
    MP_STEP64(0x111, 0xF) MP_STEP64(0x112, 0xF) MP_STEP64(0x114, 0xF) MP_STEP64(0x118, 0xF)
    MP_STEP64(0x142, 0xA) MP_STEP64(0x143, 0xC)
#undef MP_STEP64
    return v;
}

// The ready lists of the classes share one array of N slots: class c owns
// the region [region[c], region[c] + number of class-c tensors), as each
// tensor is appended once.  Appends of a round go after `end[c]` (here the
// list position past the round's own range, region included), counted by
// one 32-bit LDS counter per class.  The order of a round's appends is
// free: a tensor's fit depends only on its placed predecessors.
struct ReadyLists {
    uint16_t* slot;
    uint32_t end[kClasses];
    uint32_t* cnt;  // kClasses counters of this round's appends
};

// Decrement the pending counts of the successors among a lane's S slots:
// after a fit, a slot names a successor exactly when it holds an unplaced
// neighbour (kUnplacedBit | position; every neighbour ranked before the
// fitted tensor is placed and none ranked after it is); only those issue an
// atomic (slots masked off issue none, so no lanes pile onto one word), and
// a slot's tensor is ready exactly when the count it read was 1.  A ready
// tensor takes its list position from its class's counter (the class is
// the field of the word's count that is set).
template <int S>
__device__ __forceinline__ void release(const uint32_t (&o)[S], uint64_t* ofsz,
                                        const ReadyLists& rl, int lane) {
    uint32_t old[S];
    uint32_t* hi = reinterpret_cast<uint32_t*>(ofsz) + 1;  // the words' high halves
#pragma unroll
    for (int r = 0; r < S; ++r) {
        old[r] = 0;
        if (o[r] >= kUnplacedBit && o[r] != kNoSlot) old[r] = atomicSub(hi + 2 * (o[r] & 0xFFFFu), 1u);
    }
    uint32_t at[S];
#pragma unroll
    for (int r = 0; r < S; ++r) {
        if ((old[r] & kPendMask) == 1u) {
            const uint32_t c = (uint32_t)__builtin_ctz(old[r] >> kClassShift) >> 2;
            at[r] = rl.end[0];
            at[r] = c == 1 ? rl.end[1] : at[r];
            at[r] = c == 2 ? rl.end[2] : at[r];
            at[r] = c == 3 ? rl.end[3] : at[r];
            at[r] = c == 4 ? rl.end[4] : at[r];
            at[r] += atomicAdd(rl.cnt + c, 1u);
        }
    }
#pragma unroll
    for (int r = 0; r < S; ++r)
        if ((old[r] & kPendMask) == 1u) rl.slot[at[r]] = (uint16_t)(o[r] & 0xFFFFu);
}

// Compare-exchange of two (offset, end) slots by offset.
__device__ __forceinline__ void cex(uint32_t& oa, uint32_t& ea, uint32_t& ob, uint32_t& eb) {
    const bool sw = oa > ob;
    const uint32_t to = oa, te = ea;
    oa = sw ? ob : oa;
    ea = sw ? eb : ea;
    ob = sw ? to : ob;
    eb = sw ? te : eb;
}
// The lane's S slots sorted by offset (optimal networks: 1, 5 and 19
// comparators for 2, 4 and 8 slots); unplaced neighbours and empty slots
// (offsets at or above 2^31) end up last.
template <int S>
__device__ __forceinline__ void sort_slots(uint32_t (&o)[S], uint32_t (&e)[S]) {
#define MP_CEX(a, b) cex(o[a], e[a], o[b], e[b])
    if constexpr (S == 2) {
        MP_CEX(0, 1);
    } else if constexpr (S == 4) {
        MP_CEX(0, 1); MP_CEX(2, 3); MP_CEX(0, 2); MP_CEX(1, 3); MP_CEX(1, 2);
    } else if constexpr (S == 8) {
        MP_CEX(0, 2); MP_CEX(1, 3); MP_CEX(4, 6); MP_CEX(5, 7);
        MP_CEX(0, 4); MP_CEX(1, 5); MP_CEX(2, 6); MP_CEX(3, 7);
        MP_CEX(0, 1); MP_CEX(2, 3); MP_CEX(4, 5); MP_CEX(6, 7);
        MP_CEX(2, 4); MP_CEX(3, 5);
        MP_CEX(1, 4); MP_CEX(3, 6);
        MP_CEX(1, 2); MP_CEX(3, 4); MP_CEX(5, 6);
    }
#undef MP_CEX
}

// Lowest y >= x at which [y, y + s) meets none of the lane's ranges, the
// ranges sorted by offset: one pass suffices, since a range passed over
// either ended at or below y or was jumped past, and y only grows.
template <int S>
__device__ __forceinline__ uint32_t sweep_lowest(const uint32_t (&o)[S], const uint32_t (&e)[S],
                                                 uint32_t x, uint32_t s) {
#pragma unroll
    for (int r = 0; r < S; ++r) x = (o[r] < x + s && x < e[r]) ? e[r] : x;
    return x;
}

// BEST_FIT over the lane's ranges sorted by offset: the free gap before
// range r runs from the highest end among ranges before it to its offset;
// the smallest gap that holds s wins (lowest start among equals), else the
// space above every range.
template <int S>
__device__ __forceinline__ uint32_t sweep_best(const uint32_t (&o)[S], const uint32_t (&e)[S],
                                               uint32_t s) {
    uint32_t m = 0, bg = kNoSlot, bs = 0;
#pragma unroll
    for (int r = 0; r < S; ++r) {
        const bool placed = o[r] < kUnplacedBit;
        const bool fits = placed && o[r] >= m && o[r] - m >= s && o[r] - m < bg;
        bs = fits ? m : bs;
        bg = fits ? o[r] - m : bg;
        m = placed ? max(m, e[r]) : m;
    }
    return bg != kNoSlot ? bs : m;
}

// BEST_FIT (the tightest-gap reading of Section 2.3's "best fit"): among the
// free gaps between the placed neighbours' ranges, the smallest one that
// holds s units, the lowest start among equals; the space above every range
// only when no finite gap holds s.  A group of LANES lanes holds kBestSlots
// ranges per lane, element i = kBestSlots l + r at lane l (0 <= l < LANES)
// and slot r; the group sorts them by offset (bitonic network: slots within
// a lane, lanes by exchanges with lane l ^ d), takes running maxima of the
// ends in that order (gap before element i: [max end of elements < i,
// offset of i)) and a minimum over (gap length, gap start).  Unplaced ranges
// and empty slots (offsets at or above 2^31) sort last and bound no gap.
// Every lane of the group gets the result.
template <int LANES>
__device__ uint32_t best_fit_group(uint32_t (&o)[kBestSlots], uint32_t (&e)[kBestSlots],
                                   uint32_t s, uint32_t l) {
    constexpr int kS = kBestSlots;
    constexpr int kN = kS * LANES;
#pragma unroll
    for (int k = 2; k <= kN; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j >= 1; j >>= 1) {
            if (j < kS) {
#pragma unroll
                for (int r = 0; r < kS; ++r) {
                    const int r2 = r ^ j;
                    if (r2 > r) {
                        const bool up = ((((uint32_t)kS * l + (uint32_t)r) & (uint32_t)k) == 0);
                        const bool sw = up ? (o[r] > o[r2]) : (o[r] < o[r2]);
                        const uint32_t oa = o[r], ea = e[r];
                        o[r] = sw ? o[r2] : oa;
                        e[r] = sw ? e[r2] : ea;
                        o[r2] = sw ? oa : o[r2];
                        e[r2] = sw ? ea : e[r2];
                    }
                }
            } else {
                const int d = j / kS;  // partner lane l ^ d, same slot
                const bool lower = (l & (uint32_t)d) == 0;
#pragma unroll
                for (int r = 0; r < kS; ++r) {
                    const uint32_t po = (uint32_t)__shfl_xor((int)o[r], d, LANES);
                    const uint32_t pe = (uint32_t)__shfl_xor((int)e[r], d, LANES);
                    const bool up = ((((uint32_t)kS * l + (uint32_t)r) & (uint32_t)k) == 0);
                    const bool take = (lower == up) ? (po < o[r]) : (po > o[r]);
                    o[r] = take ? po : o[r];
                    e[r] = take ? pe : e[r];
                }
            }
        }
    }
    // running maximum of the placed ends: within the lane, then over the
    // lanes before it
    uint32_t incl[kS], run = 0;
#pragma unroll
    for (int r = 0; r < kS; ++r) {
        run = max(run, o[r] < kUnplacedBit ? e[r] : 0u);
        incl[r] = run;
    }
    uint32_t scan = run;
#pragma unroll
    for (int d = 1; d < LANES; d <<= 1) {
        const uint32_t y = (uint32_t)__shfl_up((int)scan, d, LANES);
        if (l >= (uint32_t)d) scan = max(scan, y);
    }
    uint32_t before = (uint32_t)__shfl_up((int)scan, 1, LANES);
    if (l == 0) before = 0;
    const uint32_t top = (uint32_t)__shfl((int)scan, LANES - 1, LANES);
    uint64_t best = ~0ull;
#pragma unroll
    for (int r = 0; r < kS; ++r) {
        const uint32_t pm = r == 0 ? before : max(before, incl[r - 1]);
        const bool ok = o[r] < kUnplacedBit && o[r] >= pm && o[r] - pm >= s;
        const uint64_t key = ((uint64_t)(o[r] - pm) << 32) | pm;
        best = (ok && key < best) ? key : best;
    }
#pragma unroll
    for (int d = 1; d < LANES; d <<= 1) {
        const uint32_t blo = (uint32_t)__shfl_xor((int)(uint32_t)best, d, LANES);
        const uint32_t bhi = (uint32_t)__shfl_xor((int)(uint32_t)(best >> 32), d, LANES);
        const uint64_t other = ((uint64_t)bhi << 32) | blo;
        best = other < best ? other : best;
    }
    return best != ~0ull ? (uint32_t)best : top;
}

// A tensor being fitted by a lane group: its position, size, left-list start,
// left length and neighbour count (all lanes of the group hold the same
// values).
struct Item {
    uint32_t q, s, lb, L, K;
};

// A lane without a tensor gets the spare word ofsz[N] (never placed, size
// 0) as its tensor and no neighbours.
__device__ __forceinline__ Item load_item(uint32_t q, bool has, uint32_t spare,
                                          const uint64_t* ofsz, const uint16_t* lbeg,
                                          const uint16_t* rlen) {
    Item it{spare, 0, 0, 0, 0};
    if (has) {
        it.q = q;
        it.s = (uint32_t)ofsz[q];
        it.lb = lbeg[q];
        it.L = (uint32_t)lbeg[q + 1] - it.lb;
        it.K = it.L + rlen[q];
    }
    return it;
}

// The neighbours k = S g + r (r < S) of a group's tensor, for the lane at
// position g of its group.  The neighbour sequence is the left list, then
// the right band q + 1 .. q + R.  o[r] is a placed neighbour's offset, or
// kUnplacedBit | position for an unplaced one (never overlapping, and what
// the release needs), or kNoSlot past the neighbour count; e[r] the placed
// neighbour's end.  The lane's left-list entries are consecutive bytes, read
// as aligned words (the list array is padded for the words past its end).
// LONG: the trace has long tensors (entries at or above kLongBase name one
// through the table).
template <int S, bool LONG>
__device__ __forceinline__ void gather(const Item& it, uint32_t g, const uint64_t* ofsz,
                                       const LeftLists& ll, uint32_t (&o)[S], uint32_t (&e)[S]) {
    static_assert(S == 1 || S == 2 || S == 4 || S == 8, "1, 2, 4 or 8 slots a lane");
    constexpr int kW = S == 8 ? 2 : 1;  // 32-bit words of entries a lane needs
    uint32_t id[S];
    const uint32_t k0 = g * S;
    const uint32_t s0 = it.lb + min(k0, it.L);
    const uint32_t* w32 = reinterpret_cast<const uint32_t*>(ll.ent) + (s0 >> 2);
    uint32_t by[kW];
    {
        const uint32_t b0 = w32[0], b1 = w32[1];
        by[0] = __builtin_amdgcn_alignbyte(b1, b0, s0 & 3u);
        if (kW == 2) by[kW - 1] = __builtin_amdgcn_alignbyte(w32[2], b1, s0 & 3u);
    }
    // slot r holds neighbour k0 + r: left entry r when r < lr, band position
    // rb + r when lr <= r < kr, nothing beyond (the tensor's own word is read)
    const int lr = (int)it.L - (int)k0, kr = (int)it.K - (int)k0;
    const uint32_t rb = it.q + 1u - (uint32_t)lr;
#pragma unroll
    for (int r = 0; r < S; ++r) {
        const uint32_t ent = __builtin_amdgcn_ubfe(by[r >> 2], 8 * (r & 3), 8);
        uint32_t pl = it.q - ent;
        if (LONG) {  // the table read is unconditional (in bounds), then selected
            const uint32_t lt = ll.longtab[(ent - kLongBase) & (kLongSlots - 1)];
            pl = ent >= kLongBase ? lt : pl;
        }
        const uint32_t a = r < lr ? pl : rb + (uint32_t)r;
        id[r] = r < kr ? a : it.q;
    }
    uint64_t w[S];
#pragma unroll
    for (int r = 0; r < S; ++r) w[r] = ofsz[id[r]];
#pragma unroll
    for (int r = 0; r < S; ++r) {
        const uint32_t wo = word_off(w[r]);
        o[r] = r >= kr ? kNoSlot : (wo < kUnplacedBit ? wo : (kUnplacedBit | id[r]));
        e[r] = word_end(w[r]);
    }
}

// Whole-wave placement of tensor q (all 64 lanes active, arguments uniform):
// LOWEST_FIT sweeps the neighbour sequence in chunks of kCoopChunk, lane l
// holding neighbours 8 l .. 8 l + 7 of the chunk, sorted in the lane; within
// a chunk every lane moves the candidate to the lowest start clear of its
// own ranges and the wave takes the maximum until no lane moves, and chunks
// are revisited until a full lap leaves the candidate alone.  BEST_FIT
// tensors reach here with at most kBestMaxK neighbours (more go to the
// general path): one chunk of four a lane, sorted by the wave.  Then q is
// published and its successors' pending counts are decremented.
template <bool LONG, bool BEST>
__device__ void place_wave(const Item& it, uint32_t spare, uint64_t* ofsz, const LeftLists& ll,
                           const ReadyLists& rl, int lane) {
    const uint32_t g0 = (uint32_t)lane;
    if (BEST) {
        uint32_t o[kBestSlots], e[kBestSlots];
        gather<kBestSlots, LONG>(it, g0, ofsz, ll, o, e);
        const uint32_t x = best_fit_group<kWave>(o, e, it.s, (uint32_t)lane);
        if (lane == 0) ofsz[it.q] = ((uint64_t)x << 32) | it.s;
        release<kBestSlots>(o, ofsz, rl, lane);
        return;
    }
    const uint32_t nch = (it.K + kCoopChunk - 1) / kCoopChunk;
    uint32_t o[kLaneSlots], e[kLaneSlots];
    uint32_t x = 0, clean = 0, c = 0;
    while (clean < nch) {
        if (nch > 1 || c == 0) {
            gather<kLaneSlots, LONG>(it, c * kWave + g0, ofsz, ll, o, e);
            sort_slots<kLaneSlots>(o, e);
        }
        bool moved = false;
        while (true) {
            const uint32_t xn = wave_max_u32(sweep_lowest<kLaneSlots>(o, e, x, it.s));
            if (xn == x) break;
            x = xn;
            moved = true;
        }
        clean = moved ? 1u : clean + 1u;
        c = (c + 1 == nch) ? 0u : c + 1;
    }
    if (lane == 0) ofsz[it.q] = ((uint64_t)x << 32) | it.s;
    for (uint32_t cc = 0; cc < nch; ++cc) {
        if (nch > 1) gather<kLaneSlots, LONG>(it, cc * kWave + g0, ofsz, ll, o, e);
        release<kLaneSlots>(o, ofsz, rl, lane);
    }
}

// ------------------------------------------------------------ general path

// Loads of data other threads of the workgroup stored to global memory
// before the last l2_barrier (relaxed agent-scope atomics: served by L2,
// never by a stale line of the CU's vector cache).
__device__ __forceinline__ uint64_t l2_load64(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t l2_load32(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Barrier after which every thread's global stores of the workgroup are
// complete (the workgroup barrier alone does not wait for them).
__device__ __forceinline__ void l2_barrier() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
}

// Running maximum over the workgroup in thread order: the maximum of the
// values of the threads before this one (0 for thread 0); *all gets the
// maximum over every thread.  Two barriers.
template <int BLOCK>
__device__ __forceinline__ uint64_t block_exclusive_max(uint64_t v, uint64_t* all,
                                                        uint64_t* scratch) {
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    uint64_t inc = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint64_t y = __shfl_up(inc, o, kWave);
        if (lane >= o) inc = inc > y ? inc : y;
    }
    if (lane == kWave - 1) scratch[wid] = inc;
    __syncthreads();
    uint64_t before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < BLOCK / kWave; ++w) {
        const uint64_t t = scratch[w];
        before = (w < wid && t > before) ? t : before;
        tot = t > tot ? t : tot;
    }
    __syncthreads();
    uint64_t prev = __shfl_up(inc, 1, kWave);
    if (lane == 0) prev = 0;
    *all = tot;
    return before > prev ? before : prev;
}

// Per-trace workspace of the general path (bytes from the trace's base, n
// tensors): two copies of the list of placed tensors sorted by offset --
// offsets (u64) at 0 and 8n, ids (u32) at 16n and 20n.  The live-bytes
// difference array (n + 1 u64) uses the first copy before placement.  24n + 8
// bytes in all; the LDS path keeps its position permutation (u16) at 0.
constexpr int64_t kWsPerTensor = 24;
constexpr int64_t kWsPerTrace = 64;

__device__ __forceinline__ unsigned char* trace_ws(unsigned char* ws, int64_t lo, int64_t b) {
    return ws + kWsPerTensor * lo + kWsPerTrace * b;
}

// The greedy of Section 2.3 taken literally for one trace of n tensors
// (1 <= n <= cap_n): tensors in rank order (size desc, first asc, id asc),
// each at the lowest (or, BEST_FIT, the tightest) gap left by the placed
// tensors whose lifetimes meet its own, 64-bit offsets in bytes.  The placed
// tensors are kept sorted by offset; each step filters them by lifetime,
// takes running maxima of their ends in offset order (the gap before a range
// runs from the maximum end below it to its start) and inserts the new range
// while copying the list to its other copy.  O(n^2 / BLOCK) work per trace.
// The bound is the maximum over positions of the running sum of a
// difference array (+size at a tensor's position, -size at its reach).
// LDS: at least 16 n + 8 bytes at smem.
template <int BLOCK>
__device__ void plan_general(const int64_t* __restrict__ size, const int32_t* __restrict__ first,
                             const int32_t* __restrict__ last, int64_t lo, int n, bool best,
                             unsigned char* smem, unsigned char* tws, uint64_t* red64,
                             int64_t* __restrict__ offset_out, uint64_t* peak, uint64_t* bound) {
    const int tid = threadIdx.x;
    int m = 1;
    while (m < n) m <<= 1;
    uint64_t* soff0 = reinterpret_cast<uint64_t*>(tws);
    uint64_t* soff1 = reinterpret_cast<uint64_t*>(tws + 8 * (size_t)n);
    uint32_t* sidx0 = reinterpret_cast<uint32_t*>(tws + 16 * (size_t)n);
    uint32_t* sidx1 = reinterpret_cast<uint32_t*>(tws + 20 * (size_t)n);

    // ---- live-bytes bound: positions by (first, id), difference array
    {
        uint64_t* keys = reinterpret_cast<uint64_t*>(smem);
        unsigned long long* dd = reinterpret_cast<unsigned long long*>(soff0);  // n + 1 entries
        for (int i = tid; i < m; i += BLOCK)
            keys[i] = i < n ? ((uint64_t)(uint32_t)first[lo + i] << 32) | (uint32_t)i : ~0ull;
        for (int i = tid; i <= n; i += BLOCK) dd[i] = 0ull;
        l2_barrier();
        bitonic_sort_u64<BLOCK>(keys, m);
        for (int q = tid; q < n; q += BLOCK) {
            const uint32_t id = (uint32_t)keys[q];
            const uint32_t l = (uint32_t)last[lo + id];
            int a = q + 1, z = n;  // reach: first position born after l
            while (a < z) {
                const int mid = (a + z) >> 1;
                if ((uint32_t)(keys[mid] >> 32) <= l) a = mid + 1;
                else z = mid;
            }
            const unsigned long long s = (unsigned long long)size[lo + id];
            atomicAdd(dd + q, s);
            atomicAdd(dd + a, 0ull - s);
        }
        l2_barrier();
        const int chunk = (n + BLOCK - 1) / BLOCK;
        const int a0 = min(n, tid * chunk), a1 = min(n, a0 + chunk);
        uint64_t part = 0;
        for (int i = a0; i < a1; ++i) part += l2_load64(reinterpret_cast<uint64_t*>(dd) + i);
        uint64_t tot;
        uint64_t run = block_exclusive_sum<BLOCK, uint64_t>(part, &tot, red64);
        uint64_t lm = 0;
        for (int i = a0; i < a1; ++i) {
            run += l2_load64(reinterpret_cast<uint64_t*>(dd) + i);
            lm = lm > run ? lm : run;
        }
        *bound = block_reduce<BLOCK>(lm, OpMax<uint64_t>(), red64);
    }

    // ---- rank order: a bitonic sort of the ids with the rank comparison
    uint64_t* sz = reinterpret_cast<uint64_t*>(smem);                       // 8 n
    int32_t* fs = reinterpret_cast<int32_t*>(smem + 8 * (size_t)n);        // 4 n
    uint16_t* ord = reinterpret_cast<uint16_t*>(smem + 12 * (size_t)n);    // m <= 2 n
    for (int i = tid; i < n; i += BLOCK) {
        sz[i] = (uint64_t)size[lo + i];
        fs[i] = first[lo + i];
    }
    for (int i = tid; i < m; i += BLOCK) ord[i] = i < n ? (uint16_t)i : (uint16_t)0xFFFFu;
    __syncthreads();
    auto before = [&](uint32_t a, uint32_t c) {  // does id a rank before id c? (pads last)
        if (a == 0xFFFFu) return false;
        if (c == 0xFFFFu) return true;
        if (sz[a] != sz[c]) return sz[a] > sz[c];
        if (fs[a] != fs[c]) return fs[a] < fs[c];
        return a < c;
    };
    for (int k = 2; k <= m; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < (m >> 1); i += BLOCK) {
                const int a = ((i & ~(j - 1)) << 1) | (i & (j - 1));
                const int c = a | j;
                const uint32_t va = ord[a], vc = ord[c];
                const bool up = (a & k) == 0;
                if (before(vc, va) == up) {
                    ord[a] = (uint16_t)vc;
                    ord[c] = (uint16_t)va;
                }
            }
            __syncthreads();
        }
    }

    // ---- placement, one tensor a step
    uint64_t pk = 0;
    for (int k = 0; k < n; ++k) {
        const uint32_t t = ord[k];
        const uint64_t st = sz[t];
        const int32_t ft = first[lo + t], lt = last[lo + t];
        const uint64_t* so = (k & 1) ? soff1 : soff0;
        const uint32_t* si = (k & 1) ? sidx1 : sidx0;
        uint64_t* no = (k & 1) ? soff0 : soff1;
        uint32_t* ni = (k & 1) ? sidx0 : sidx1;
        const int chunk = (k + BLOCK - 1) / BLOCK;  // k tensors are placed
        const int e0 = min(k, tid * chunk), e1 = min(k, e0 + chunk);
        auto meets = [&](uint32_t id) { return first[lo + id] <= lt && ft <= last[lo + id]; };
        uint64_t hi = 0;  // highest end among this thread's ranges that meet t
        for (int e = e0; e < e1; ++e) {
            const uint32_t id = l2_load32(si + e);
            if (meets(id)) {
                const uint64_t en = l2_load64(so + e) + sz[id];
                hi = hi > en ? hi : en;
            }
        }
        uint64_t top;
        uint64_t run = block_exclusive_max<BLOCK>(hi, &top, red64);
        uint64_t cand = ~0ull, cgap = ~0ull;  // this thread's choice among its gaps
        for (int e = e0; e < e1; ++e) {
            const uint32_t id = l2_load32(si + e);
            if (!meets(id)) continue;
            const uint64_t o = l2_load64(so + e);
            if (o >= run && o - run >= st) {
                if (!best) {
                    if (cand == ~0ull) cand = run;
                } else if (o - run < cgap) {
                    cgap = o - run;
                    cand = run;
                }
            }
            const uint64_t en = o + sz[id];
            run = run > en ? run : en;
        }
        uint64_t x;
        if (!best) {
            x = block_reduce<BLOCK>(cand, OpMin<uint64_t>(), red64);
        } else {
            const uint64_t g = block_reduce<BLOCK>(cgap, OpMin<uint64_t>(), red64);
            x = block_reduce<BLOCK>(cgap == g ? cand : ~(uint64_t)0, OpMin<uint64_t>(), red64);
        }
        if (x == ~0ull) x = top;  // no gap holds t: above every range
        pk = pk > x + st ? pk : x + st;
        if (tid == 0) offset_out[lo + t] = (int64_t)x;
        // the list with t inserted before the first range starting at or above x
        for (int e = e0; e < e1; ++e) {
            const uint64_t o = l2_load64(so + e);
            const uint32_t id = l2_load32(si + e);
            const int d = e + (o >= x ? 1 : 0);
            no[d] = o;
            ni[d] = id;
            if (o >= x && (e == 0 || l2_load64(so + e - 1) < x)) {
                no[e] = x;
                ni[e] = t;
            }
        }
        if (tid == 0 && (k == 0 || l2_load64(so + k - 1) < x)) {
            no[k] = x;
            ni[k] = t;
        }
        l2_barrier();
    }
    *peak = pk;
}

// LDS byte offsets of the regions of the LDS path (N = tensor slots):
//   A [8N+8]   first (i32) and live-bytes deltas (u32, from 4N)
//              -> fill: cursors (u16, at 0), predecessor counts (u16, at
//                 2N+4), sizes in units (u32, at 4N+8)
//              -> placement words ofsz[N + 1]
//   F [2N+4]   band lengths (u16), kept for placement
//   E [2N+4]   left-list starts (u16, N + 1 of them)
//   R [2N+4]   reach histogram (packed u16) -> band starts -> ready lists
//   T [cap+16] left-list entries (u8)
// The u64 sort keys of an unsorted trace use the space from 0 before the
// reach pass, and the general path uses all of it (16N + 8 at least).
struct BatchLds {
    size_t a, f, e, r, t, total;
};
__host__ __device__ inline BatchLds batch_lds(size_t N, size_t cap) {
    BatchLds L{};
    const size_t w16 = (2 * N + 4 + 3) & ~(size_t)3;  // N + 1 u16 entries, 4-byte multiple
    L.a = 0;
    L.f = 8 * N + 8;
    L.e = L.f + w16;
    L.r = L.e + w16;
    L.t = L.r + w16;
    L.total = (L.t + cap + 16 + 15) & ~(size_t)15;
    return L;
}

// The k-th item of this thread, tid + k * BLOCK, computed where it is used:
// the thread index goes through an empty asm so that the compiler cannot
// keep the items of one phase alive into the next (it spilled them to
// scratch memory rather than recompute them with one addition).
template <int BLOCK>
__device__ __forceinline__ int item_index(int k) {
    int t = (int)threadIdx.x;
    asm volatile("" : "+v"(t));
    return t + k * BLOCK;
}

template <int BLOCK, int ITEMS, bool BEST>
__global__ __launch_bounds__(BLOCK, BEST ? 4 : (ITEMS <= 4 ? 6 : 4)) void plan_batch_kernel(
    const int64_t* __restrict__ begin, const int32_t* __restrict__ num_ops,
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, int64_t n_tensors, int32_t cap_n, int32_t cap_lists,
    unsigned char* __restrict__ ws, int64_t* __restrict__ offset_out,
    int64_t* __restrict__ peak_out, int64_t* __restrict__ lb_out, int32_t* __restrict__ status) {
    const uint64_t t_start = wall_clock64();
    constexpr bool best = BEST;  // BEST_FIT: one lane up to 8 neighbours, else the whole wave
    extern __shared__ __align__(16) unsigned char smem[];
    // static LDS: at most kStaticLds bytes (checked at launch), or four
    // workgroups of a 2000-tensor trace no longer fit a CU
    __shared__ uint64_t red[BLOCK / kWave];
    __shared__ uint64_t red3[3][BLOCK / kWave];  // ingest reductions, then the prefix pass's
    uint32_t(*red32)[BLOCK / kWave] = reinterpret_cast<uint32_t(*)[BLOCK / kWave]>(&red3[0][0]);
    __shared__ uint32_t nready[3][kClasses];  // appended in rounds r % 3, per class
    __shared__ unsigned long long ncls64;     // tensors per ready class 0-3 (16-bit fields)
    __shared__ unsigned long long seeds64;    // ... without predecessors
    __shared__ uint32_t ncls_w, seeds_w;      // ... of class 4
    __shared__ uint16_t longtab[kLongSlots];  // positions of the long tensors
    __shared__ uint32_t nlong;

    const size_t N = (size_t)cap_n;
    const BatchLds R = batch_lds(N, (size_t)cap_lists);
    int32_t* fst = reinterpret_cast<int32_t*>(smem + R.a);
    uint32_t* live = reinterpret_cast<uint32_t*>(smem + R.a + 4 * N);
    uint32_t* cursor = reinterpret_cast<uint32_t*>(smem + R.a);
    uint32_t* pend = reinterpret_cast<uint32_t*>(smem + R.a + 2 * N + 4);
    uint32_t* su = reinterpret_cast<uint32_t*>(smem + R.a + 4 * N + 8);
    uint64_t* ofsz = reinterpret_cast<uint64_t*>(smem + R.a);
    uint64_t* keys = reinterpret_cast<uint64_t*>(smem);
    uint16_t* rlen = reinterpret_cast<uint16_t*>(smem + R.f);
    uint16_t* lbeg = reinterpret_cast<uint16_t*>(smem + R.e);
    uint32_t* hist = reinterpret_cast<uint32_t*>(smem + R.r);
    uint16_t* bstart = reinterpret_cast<uint16_t*>(smem + R.r);
    uint16_t* readyq = reinterpret_cast<uint16_t*>(smem + R.r);
    uint8_t* lents = smem + R.t;
    uint32_t* scratch = reinterpret_cast<uint32_t*>(red);

    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    MP_STAMP(0);
    if (tid == 0) {
        for (int r = 0; r < 3; ++r)
            for (int c = 0; c < kClasses; ++c) nready[r][c] = 0;
        ncls_w = seeds_w = 0;
        ncls64 = seeds64 = 0;
        nlong = 0;
    }
    const int64_t lo = begin[b], hi = begin[b + 1];
    const int32_t n_ops = num_ops[b];
    if (lo < 0 || hi < lo || hi > n_tensors || n_ops < 0 || hi - lo > cap_n) {
        if (tid == 0) raise_status(status, MP_EINVAL);
        return;
    }
    const int n = (int)(hi - lo);
    unsigned char* tws = trace_ws(ws, lo, b);
    uint16_t* perm = reinterpret_cast<uint16_t*>(tws);  // ids by position (unsorted traces)

    // ---- ingest + checks (ids owned strided: i = tid + k * BLOCK).  The
    // sizes and last ops of a sorted trace stay in registers for the band
    // pass; later phases reload what they need (from L2).
    uint32_t flags = 0;  // bit 0: invalid tensor, bit 1: first not sorted
    uint64_t orv = 0, sum = 0;
    int64_t sz_r[ITEMS];
    int32_t la_r[ITEMS];
    // every load is issued before any is used: indices are clamped into
    // the trace (n >= 1 here), so the loads need no branch around them
    int32_t fi_r[ITEMS], fp_r[ITEMS];
    if (n > 0) {
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int i = min(item_index<BLOCK>(k), n - 1);
            sz_r[k] = size[lo + i];
            fi_r[k] = first[lo + i];
            la_r[k] = last[lo + i];
            fp_r[k] = first[lo + (i > 0 ? i - 1 : 0)];
        }
    }
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int i = item_index<BLOCK>(k);
        if (i < n) {
            const int64_t s = sz_r[k];
            const int32_t f = fi_r[k], l = la_r[k];
            if (i > 0 && fp_r[k] > f) flags |= 2u;
            if (s <= 0 || f < 0 || f > l || l >= n_ops) flags |= 1u;
            if (s > 0) {
                orv |= (uint64_t)s;
                sum = sat_add(sum, (uint64_t)s);
            }
            fst[i] = f;
        } else {
            sz_r[k] = 0;
            la_r[k] = 0;
        }
    }
    // one combined reduction of the flags, the OR and the saturating sum
    uint64_t or_all, total;
    {
        const int lane = tid & (kWave - 1), wid = tid / kWave;
        flags = wave_reduce(flags, OpOr<uint32_t>());
        orv = wave_reduce(orv, OpOr<uint64_t>());
        sum = wave_reduce(sum, OpSatAdd());
        if (lane == 0) {
            red3[0][wid] = flags;
            red3[1][wid] = orv;
            red3[2][wid] = sum;
        }
        __syncthreads();
        flags = 0;
        or_all = 0;
        total = 0;
#pragma unroll
        for (int w = 0; w < BLOCK / kWave; ++w) {
            flags |= (uint32_t)red3[0][w];
            or_all |= red3[1][w];
            total = sat_add(total, red3[2][w]);
        }
    }
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
    bool general = (total >> sh) > kFastMaxUnits;
    // sizes in units (below 2^31 unless general), kept instead of the bytes
    uint32_t su_r[ITEMS];
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) su_r[k] = (uint32_t)((uint64_t)sz_r[k] >> sh);
    const bool unsorted = (flags & 2u) != 0;
    auto id_of = [&](int q) { return unsorted ? (int)perm[q] : q; };  // position -> id

    uint32_t live_max = 0, n_pairs = 0;
    if (!general) {
        // ---- position order (first, id); recorded traces are normally sorted already
        if (unsorted) {
            int m = 1;
            while (m < n) m <<= 1;
            for (int i = tid; i < m; i += BLOCK)
                keys[i] = (i < n) ? (((uint64_t)(uint32_t)first[lo + i] << 32) | (uint32_t)i) : ~0ull;
            __syncthreads();
            bitonic_sort_u64<BLOCK>(keys, m);
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                const int q = item_index<BLOCK>(k);
                if (q < n) perm[q] = (uint16_t)(keys[q] & 0xFFFFu);
            }
            l2_barrier();  // the keys are dead: first[] goes back in position order
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                const int q = item_index<BLOCK>(k);
                if (q < n) fst[q] = first[lo + perm[q]];
            }
        }
        for (int i = tid; i <= n; i += BLOCK) live[i] = 0;
        for (int i = tid; i <= (n >> 1); i += BLOCK) hist[i] = 0;
        __syncthreads();
        MP_STAMP(2);

        // ---- reach, band lengths, live-bytes deltas, reach histogram, long
        // tensors.  The reach is the first position past q whose first op is
        // after last[q].  When the ops are no more than the tensor slots (one
        // op per tensor or fewer, as recorded traces are), it is read from a
        // table over ops, P[op] = number of positions whose first op is at
        // most op, filled from the first ops in position order (P sits in the
        // left-list starts' region, unused until the prefix pass).  Otherwise
        // the next four positions are probed at once (short bands, the common
        // case, end there) and longer bands gallop from the fourth.
        const bool by_table = n_ops <= (int32_t)N + 1;
        uint16_t* ptab = lbeg;
        if (by_table) {
            // position i owns the ops [first[i], first[i + 1]) (i = -1: the ops
            // before the first first op; i = n - 1: up to the last op)
            for (int i = tid - 1; i < n; i += BLOCK) {
                const int a = i < 0 ? 0 : fst[i];
                const int z = i + 1 < n ? fst[i + 1] : n_ops;
                for (int op = a; op < z; ++op) ptab[op] = (uint16_t)(i + 1);
            }
            __syncthreads();
        }
        int32_t rch[ITEMS];
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int q = item_index<BLOCK>(k);
            rch[k] = q + 1;
            if (q < n) {
                const int32_t l = last[lo + (unsorted ? (int)perm[q] : q)];
                if (by_table) {
                    rch[k] = ptab[l];
                } else {
                    const int32_t f1 = q + 1 < n ? fst[q + 1] : INT32_MAX;
                    const int32_t f2 = q + 2 < n ? fst[q + 2] : INT32_MAX;
                    const int32_t f3 = q + 3 < n ? fst[q + 3] : INT32_MAX;
                    const int32_t f4 = q + 4 < n ? fst[q + 4] : INT32_MAX;
                    rch[k] = q + 1 + (f1 <= l) + (f2 <= l) + (f3 <= l) + (f4 <= l);
                }
            }
        }
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int q = item_index<BLOCK>(k);
            if (q < n) {
                const int32_t l = last[lo + (unsorted ? (int)perm[q] : q)];
                const uint32_t sq =
                    unsorted ? (uint32_t)((uint64_t)size[lo + perm[q]] >> sh) : su_r[k];
                int a = rch[k];
                if (!by_table && a == q + 5) {  // first[q + 4] <= l: gallop on
                    int known = q + 4, step = 8, probe = q + 8;  // first[known] <= l
                    while (probe < n && fst[probe] <= l) {
                        known = probe;
                        step <<= 1;
                        probe = q + step;
                    }
                    a = known + 1;
                    int z = probe < n ? probe : n;
                    while (a < z) {
                        const int mid = (a + z) >> 1;
                        if (fst[mid] <= l) a = mid + 1;
                        else z = mid;
                    }
                }
                rlen[q] = (uint16_t)(a - q - 1);
                atomicAdd(&live[q], sq);
                atomicAdd(&live[a], 0u - sq);
                packed_add(hist, (uint32_t)a, 1u);
                if ((uint32_t)(a - q - 1) > kMaxDist) {  // reaches beyond a one-byte distance
                    const uint32_t slot = atomicAdd(&nlong, 1u);
                    if (slot < kLongSlots) longtab[slot] = (uint16_t)q;
                }
            }
        }
        __syncthreads();
        MP_STAMP(3);
        general = nlong > kLongSlots;
    }
    if (!general) {
        // ---- one prefix pass over positions j (contiguous chunk per thread):
        //   band start      = sum of band lengths before j        (pair index base)
        //   left-list start = sum over i < j of #{q : q < i < reach[q]}
        //                   = j(j-1)/2 - j * H(<j) + sum_{r<j} r * hist[r],
        //     since position i has i - #{q : reach[q] <= i} left neighbours;
        //   live bytes      = running sum of the deltas (its maximum is the bound).
        // The three integer sums share one 64-bit word: band (24 bits, at most
        // n(n-1)/2), hist count (13 bits, at most n) and r * hist (25 bits).
        uint32_t kmax = 0;
        {
            // even-sized chunks: both halves of a packed word stay with one thread
            const int chunk = (((n + BLOCK - 1) / BLOCK) + 1) & ~1;
            const int a0 = min(n, tid * chunk), a1 = min(n, a0 + chunk);
            auto pack = [](uint32_t bl, uint32_t h, uint32_t j) {
                return ((uint64_t)bl << 38) | ((uint64_t)h << 25) | (uint64_t)(h * j);
            };
            uint64_t ps = 0;
            uint32_t ds = 0;
            for (int i = a0; i < a1; ++i) {
                ps += pack(rlen[i], packed_get(hist, (uint32_t)i), (uint32_t)i);
                ds += live[i];
            }
            // both prefix sums over the workgroup at once (wave scans by DPP,
            // one barrier), then both maxima (one more)
            const int lane = tid & (kWave - 1), wid = tid / kWave;
            const uint64_t pin = wave_inclusive_sum64_dpp(ps);
            const uint32_t din = wave_inclusive_sum_dpp(ds);
            if (lane == kWave - 1) {
                red[wid] = pin;
                red32[0][wid] = din;
            }
            __syncthreads();
            uint64_t prun = pin - ps, ptot = 0;
            uint32_t drun = din - ds;
#pragma unroll
            for (int w = 0; w < BLOCK / kWave; ++w) {
                const uint64_t t = red[w];
                const uint32_t u = red32[0][w];
                prun += w < wid ? t : 0ull;
                drun += w < wid ? u : 0u;
                ptot += t;
            }
            uint32_t lm = 0;
            uint16_t* cursor16 = reinterpret_cast<uint16_t*>(cursor);
            for (int i = a0; i < a1; ++i) {
                const uint32_t bl = rlen[i], h = packed_get(hist, (uint32_t)i), dl = live[i];
                const uint32_t hb = (uint32_t)(prun >> 25) & 0x1FFFu;
                const uint32_t rh = (uint32_t)prun & 0x1FFFFFFu;
                const uint32_t ls = (uint32_t)(i * (i - 1) / 2) - (uint32_t)i * hb + rh;
                const uint32_t Li = (uint32_t)i - hb - h;  // left neighbours of position i
                kmax = max(kmax, Li + bl);
                bstart[i] = (uint16_t)(prun >> 38);  // over hist[i], already read
                lbeg[i] = (uint16_t)ls;
                cursor16[i] = (uint16_t)ls;
                drun += dl;
                lm = lm > drun ? lm : drun;
                prun += pack(bl, h, (uint32_t)i);
            }
            n_pairs = (uint32_t)(ptot >> 38);
            if (tid == 0) {
                bstart[n] = (uint16_t)n_pairs;
                lbeg[n] = (uint16_t)n_pairs;
            }
            const uint32_t wl = wave_max_u32(lm), wk = wave_max_u32(kmax);
            if (lane == 0) {
                red32[1][wid] = wl;
                red32[2][wid] = wk;
            }
            __syncthreads();
            live_max = 0;
            kmax = 0;
#pragma unroll
            for (int w = 0; w < BLOCK / kWave; ++w) {
                live_max = max(live_max, red32[1][w]);
                kmax = max(kmax, red32[2][w]);
            }
        }
        general = n_pairs > (uint32_t)cap_lists || (best && kmax > kBestMaxK);
    }
    if (general) {
        __syncthreads();
        uint64_t pk = 0, bound = 0;
        plan_general<BLOCK>(size, first, last, lo, n, best, smem, tws, red, offset_out, &pk,
                            &bound);
        if (tid == 0) {
            peak_out[b] = (int64_t)pk;
            if (lb_out) lb_out[b] = (int64_t)bound;
        }
        return;
    }
    MP_STAMP(4);

    // ---- sizes in units and zero predecessor counts (over first[] and the
    // deltas, both dead)
    for (int i = tid; i <= (n >> 1); i += BLOCK) pend[i] = 0;
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = item_index<BLOCK>(k);
        if (q < n) su[q] = unsorted ? (uint32_t)((uint64_t)size[lo + perm[q]] >> sh) : su_r[k];
    }
    __syncthreads();

    // ---- left lists and pending predecessor counts, balanced over the pairs:
    // pair index p -> (q, j), j = q + 1 + (p - band start of q)
    {
        const uint32_t per = (n_pairs + BLOCK - 1) / BLOCK;
        const uint32_t p_lo = min(n_pairs, (uint32_t)tid * per), p_hi = min(n_pairs, p_lo + per);
        if (p_lo < p_hi) {
            int a = 0, z = n;  // last position whose band starts at or before p_lo
            while (a < z) {
                const int mid = (a + z + 1) >> 1;
                if (bstart[mid] <= p_lo) a = mid;
                else z = mid - 1;
            }
            int q = a;
            uint32_t base = bstart[q], nxt = bstart[q + 1];
            uint32_t sq = su[q];
            for (uint32_t p = p_lo; p < p_hi; ++p) {
                while (nxt <= p) {
                    ++q;
                    base = nxt;
                    nxt = bstart[q + 1];
                    sq = su[q];
                }
                const uint32_t j = (uint32_t)q + 1 + (p - base);
                const uint32_t d = j - (uint32_t)q;
                uint32_t ent = d;
                if (d > kMaxDist) {  // q is long: its slot in the table
                    uint32_t s = 0;
#pragma nounroll
                    while (s + 1 < kLongSlots && longtab[s] != (uint16_t)q) ++s;
                    ent = kLongBase + s;
                }
                lents[packed_add(cursor, j, 1u)] = (uint8_t)ent;
                packed_add(pend, sq >= su[j] ? j : (uint32_t)q, 1u);  // j ranks after q?
            }
        }
    }
    __syncthreads();

    // ---- placement words (pending count and ready class while unplaced),
    // class regions, and the tensors without predecessors as seeds.  The
    // words overwrite the fill's arrays: read everything first.  Per lane,
    // the counts per class of its tensors and of its seeds go in 10-bit
    // fields (classes 0-2 in one word, 3-4 in another); one wave scan of the
    // seed counts and one reservation per wave place the seeds.
    const int lane_id = tid & (kWave - 1);
    uint64_t w_r[ITEMS];
    uint32_t cls_r[ITEMS];
    uint32_t tlo = 0, thi = 0, slo = 0, shi = 0, sb4 = 0;
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = item_index<BLOCK>(k);
        cls_r[k] = 7;  // no tensor
        w_r[k] = 0;
        if (q < n) {
            const uint32_t K = (uint32_t)lbeg[q + 1] - lbeg[q] + rlen[q];
            const uint32_t c = ready_class(K, best);
            const uint32_t pc = packed_get(pend, (uint32_t)q);
            w_r[k] = ((uint64_t)(kUnplacedBit | class_bits(c) | pc) << 32) | su[q];
            cls_r[k] = pc == 0 ? c + 8 : c;  // +8: a seed
            const uint32_t f = 1u << (10u * (c < 3u ? c : c - 3u));
            tlo += c < 3u ? f : 0u;
            thi += c < 3u ? 0u : f;
            slo += (c < 3u && pc == 0) ? f : 0u;
            shi += (c >= 3u && pc == 0) ? f : 0u;
        }
    }
    {
        const uint32_t tl = wave_inclusive_sum_dpp(tlo), th = wave_inclusive_sum_dpp(thi);
        const uint32_t sl = wave_inclusive_sum_dpp(slo), sh2 = wave_inclusive_sum_dpp(shi);
        const uint32_t Tl = (uint32_t)__builtin_amdgcn_readlane((int)tl, 63);
        const uint32_t Th = (uint32_t)__builtin_amdgcn_readlane((int)th, 63);
        const uint32_t Sl = (uint32_t)__builtin_amdgcn_readlane((int)sl, 63);
        const uint32_t Sh = (uint32_t)__builtin_amdgcn_readlane((int)sh2, 63);
        auto pack4 = [](uint32_t l, uint32_t h) {  // classes 0-3 as 16-bit fields
            return (unsigned long long)(l & 0x3FFu) | ((unsigned long long)((l >> 10) & 0x3FFu) << 16) |
                   ((unsigned long long)(l >> 20) << 32) | ((unsigned long long)(h & 0x3FFu) << 48);
        };
        uint32_t b0 = 0, b1 = 0, b4 = 0;
        if (lane_id == 0) {
            atomicAdd(&ncls64, pack4(Tl, Th));
            if (Th >> 10) atomicAdd(&ncls_w, Th >> 10);
            const unsigned long long base = atomicAdd(&seeds64, pack4(Sl, Sh));
            b0 = (uint32_t)base;
            b1 = (uint32_t)(base >> 32);
            if (Sh >> 10) b4 = atomicAdd(&seeds_w, Sh >> 10);
        }
        b0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)b0);
        b1 = (uint32_t)__builtin_amdgcn_readfirstlane((int)b1);
        b4 = (uint32_t)__builtin_amdgcn_readfirstlane((int)b4);
        const uint32_t xl = sl - slo, xh = sh2 - shi;  // seeds of the lanes before
        // this lane's next seed position in each class list (region added below)
        tlo = b0 & 0xFFFFu; tlo += xl & 0x3FFu;
        thi = (b0 >> 16) + ((xl >> 10) & 0x3FFu);
        slo = (b1 & 0xFFFFu) + (xl >> 20);
        shi = (b1 >> 16) + (xh & 0x3FFu);
        sb4 = b4 + (xh >> 10);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = item_index<BLOCK>(k);
        if (q < n) ofsz[q] = w_r[k];
    }
    const uint32_t spare = (uint32_t)N;  // ofsz[N]: never placed, size 0
    if (tid == 0) ofsz[spare] = (uint64_t)kUnplacedBit << 32;
    uint32_t region[kClasses];
    {
        const unsigned long long nc = ncls64;
        region[0] = 0;
        region[1] = (uint32_t)nc & 0xFFFFu;
        region[2] = region[1] + ((uint32_t)(nc >> 16) & 0xFFFFu);
        region[3] = region[2] + ((uint32_t)(nc >> 32) & 0xFFFFu);
        region[4] = region[3] + (uint32_t)(nc >> 48);
    }
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = item_index<BLOCK>(k);
        if (q < n && cls_r[k] >= 8u) {
            const uint32_t c = cls_r[k] & 7u;
            uint32_t a = tlo;
            a = c == 1 ? thi : a;
            a = c == 2 ? slo : a;
            a = c == 3 ? shi : a;
            a = c == 4 ? sb4 : a;
            readyq[region[c] + a] = (uint16_t)q;
            tlo += c == 0 ? 1u : 0u;
            thi += c == 1 ? 1u : 0u;
            slo += c == 2 ? 1u : 0u;
            shi += c == 3 ? 1u : 0u;
            sb4 += c == 4 ? 1u : 0u;
        }
    }
    __syncthreads();
    MP_STAMP(5);

    // ---- placement in rounds (Kahn's order over the predecessor DAG): round
    // r fits every tensor released in round r - 1 -- all of its predecessors
    // are placed, and no two of them intersect.  The round's tensors are
    // dealt over the workgroup's lanes in one pass, eight-lane groups first
    // (neighbour counts 33..64), then quads (17..32), pairs (9..16) and single
    // lanes (up to 8), so every group is aligned; eight neighbours a lane
    // (a short round spreads them thinner: four a lane, groups twice as
    // wide).  A lane sorts its neighbours' ranges by offset and
    // sweeps them once for the lowest start clear of them; a group takes the
    // maximum over its lanes until no lane moves.  Then the word is published and the successors'
    // pending counts decremented; those reaching zero are appended for the
    // next round.  Tensors with more than 64 neighbours (under BEST_FIT, more
    // than 8) take a whole wave each, dealt over the waves.  Waves with no
    // lane in the round go straight to its barrier.  Per-round append
    // counters rotate over three slots so that one barrier per round
    // suffices.
    auto place_rounds = [&](auto long_tag) {
        constexpr bool LONG = decltype(long_tag)::value;
        const LeftLists ll{lents, longtab};
        const int lane = lane_id;
        const uint32_t wbase = (uint32_t)(tid & ~(kWave - 1));
        uint32_t bgn[kClasses] = {0, 0, 0, 0, 0};
        uint32_t end[kClasses];
        {
            const unsigned long long sd = seeds64;
#pragma unroll
            for (int c = 0; c < 4; ++c) end[c] = (uint32_t)(sd >> (16 * c)) & 0xFFFFu;
            end[kWideClass] = seeds_w;
        }
        for (int round = 0;; ++round) {
            {
                const int64_t el = (int64_t)(wall_clock64() - t_start);
                const int64_t behind = (el - kPaceSetup) / kPaceRound - round;
                if (behind >= 3) __builtin_amdgcn_s_setprio(3);
                else if (behind == 2) __builtin_amdgcn_s_setprio(2);
                else if (behind == 1) __builtin_amdgcn_s_setprio(1);
                else __builtin_amdgcn_s_setprio(0);
            }
            const uint32_t n0 = end[0] - bgn[0], n1 = end[1] - bgn[1], n2 = end[2] - bgn[2];
            const uint32_t n3 = end[3] - bgn[3], n4 = end[4] - bgn[4];
            if ((n0 | n1 | n2 | n3 | n4) == 0) break;
            if (round > n) {  // cannot happen: every round places a tensor
                if (tid == 0) raise_status(status, MP_EDEVICE);
                break;
            }
            const int cur = round % 3, nxt = (round + 1) % 3;
            if (tid == 0) {
                // a zero made here: left to the compiler it was kept in a
                // register across the loop, spilled, and reloaded every round
                uint32_t z;
                asm volatile("v_mov_b32 %0, 0" : "=v"(z));
#pragma unroll
                for (int c = 0; c < kClasses; ++c) nready[nxt][c] = z;
            }
            const ReadyLists rl{readyq,
                                {region[0] + end[0], region[1] + end[1], region[2] + end[2],
                                 region[3] + end[3], region[4] + end[4]},
                                nready[cur]};
            // lane space of the round at S slots a lane: class c takes groups
            // of (8 / S) << c lanes, [0, a3) class 3, [a3, a2) class 2,
            // [a2, a1) class 1, [a1, tot) class 0 (aligned: largest first).
            // A round that fits the workgroup's lanes at four slots a lane is
            // spread that way (shorter passes where the rounds are short; one
            // or two a lane measured slower, the group maxima growing);
            // BEST_FIT keeps eight.
            auto run = [&](auto slots_tag) {
                constexpr int S = decltype(slots_tag)::value;
                constexpr uint32_t M = 8u / S;
                const uint32_t a3 = 8u * M * n3, a2 = a3 + 4u * M * n2, a1 = a2 + 2u * M * n1;
                const uint32_t tot = a1 + M * n0;
                for (uint32_t pass = 0; pass < tot; pass += BLOCK) {
                    if (pass + wbase >= tot) break;  // wave-uniform: nothing for this wave
                    const uint32_t gl = pass + (uint32_t)tid;
                    uint32_t c, lg;  // class, log2 of its group width
                    if (gl < a3) {
                        c = 3; lg = 3;
                    } else if (gl < a2) {
                        c = 2; lg = 2;
                    } else if (gl < a1) {
                        c = 1; lg = 1;
                    } else {
                        c = 0; lg = 0;
                    }
                    lg += (uint32_t)__builtin_ctz(M);
                    const uint32_t G = 1u << lg;
                    const uint32_t start = c == 3 ? 0u : (c == 2 ? a3 : (c == 1 ? a2 : a1));
                    const uint32_t idx = (gl - start) >> lg;
                    const bool has = gl < tot;
                    const uint32_t g = gl & (G - 1u);
                    uint32_t q = 0;
                    if (has) {
                        uint32_t at = region[0] + bgn[0];
                        at = c == 1 ? region[1] + bgn[1] : at;
                        at = c == 2 ? region[2] + bgn[2] : at;
                        at = c == 3 ? region[3] + bgn[3] : at;
                        q = readyq[at + idx];
                    }
                    const Item it = load_item(q, has, spare, ofsz, lbeg, rlen);
                    uint32_t o[S], e[S];
                    gather<S, LONG>(it, g, ofsz, ll, o, e);
                    sort_slots<S>(o, e);
                    uint32_t x;
                    if (best) {
                        x = sweep_best<S>(o, e, it.s);  // class 0 only: K <= 8, one lane
                    } else {
                        x = group_max_u32(sweep_lowest<S>(o, e, 0u, it.s), G);
                        if (M > 1 || __ballot(G > 1u)) {
                            while (true) {
                                const uint32_t xn = group_max_u32(sweep_lowest<S>(o, e, x, it.s), G);
                                if (!__ballot(xn != x)) break;
                                x = xn;
                            }
                        }
                    }
                    if (has && g == 0) ofsz[it.q] = ((uint64_t)x << 32) | it.s;
                    release<S>(o, ofsz, rl, lane);
                }
            };
            const uint32_t t8 = n0 + 2u * n1 + 4u * n2 + 8u * n3;  // lanes at eight slots
            if (best || 2u * t8 > (uint32_t)BLOCK) run(std::integral_constant<int, 8>{});
            else run(std::integral_constant<int, 4>{});
            // more neighbours than eight lanes hold: the whole wave each, dealt
            // over the waves
            for (uint32_t i0 = bgn[4] + (wbase / kWave); i0 < end[4]; i0 += BLOCK / kWave) {
                const uint32_t qw = readyq[region[4] + i0];
                const Item iw = load_item(qw, true, spare, ofsz, lbeg, rlen);
                const Item one{(uint32_t)__builtin_amdgcn_readfirstlane((int)iw.q),
                               (uint32_t)__builtin_amdgcn_readfirstlane((int)iw.s),
                               (uint32_t)__builtin_amdgcn_readfirstlane((int)iw.lb),
                               (uint32_t)__builtin_amdgcn_readfirstlane((int)iw.L),
                               (uint32_t)__builtin_amdgcn_readfirstlane((int)iw.K)};
                place_wave<LONG, best>(one, spare, ofsz, ll, rl, lane);
            }
            __syncthreads();
            uint32_t added[kClasses];
#pragma unroll
            for (int c = 0; c < kClasses; ++c) added[c] = nready[cur][c];
#pragma unroll
            for (int c = 0; c < kClasses; ++c) bgn[c] = end[c];
#pragma unroll
            for (int c = 0; c < kClasses; ++c) end[c] += added[c];
        }
    };
    if (nlong) place_rounds(std::true_type{});
    else place_rounds(std::false_type{});
    __syncthreads();
    MP_STAMP(6);

    // ---- outputs
    uint32_t pk = 0;
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = item_index<BLOCK>(k);
        if (q < n) {
            const uint64_t w = ofsz[q];
            offset_out[lo + id_of(q)] = (int64_t)((uint64_t)word_off(w) << sh);
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

// Static LDS of the kernel, rounded up (the per-workgroup budget minus this
// is dynamic).
constexpr size_t kStaticLds = 512;

template <int BLOCK, int ITEMS, bool BEST>
hipError_t launch_items(const BatchArgs& a, const BatchShape& s, hipStream_t st) {
    auto kern = plan_batch_kernel<BLOCK, ITEMS, BEST>;
    hipFuncAttributes fa{};
    hipError_t e = hipFuncGetAttributes(&fa, (const void*)kern);
    if (e != hipSuccess) return e;
    if (fa.sharedSizeBytes > kStaticLds) return hipErrorInvalidConfiguration;  // LDS budget broken
    e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)s.lds_bytes);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)a.n_traces), dim3(BLOCK), s.lds_bytes, st,
                       a.begin, a.num_ops, a.size, a.first, a.last, a.n_tensors, s.cap_n,
                       s.cap_pairs, static_cast<unsigned char*>(a.workspace), a.offset_out,
                       a.peak_out, a.lb_out, a.status);
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

// LDS per workgroup: about 14 bytes per tensor slot plus one byte per list
// entry, in the smallest budget of {1/4, 1/3, 1/2, all} of a CU's 160 KiB
// that gives every pair of a trace of max_trace_len tensors a slot, or at
// least 4 per tensor (and at least 2 per tensor always: the sort keys of an
// unsorted trace and the general path's 16 bytes per tensor use the same
// space); the list capacity is whatever that budget leaves.  List starts are
// u16: at most 65520 entries.  A trace with more pairs than the capacity
// takes the general path.
BatchShape batch_shape(int64_t max_trace_len) {
    BatchShape s{};
    if (max_trace_len < 0 || max_trace_len > MP_BATCH_MAX_TRACE_LEN) return s;
    const int64_t N = max_trace_len < 1 ? 1 : max_trace_len;
    int64_t want = N * (N - 1) / 2;
    if (want > 4 * N) want = 4 * N;
    if (want < 2 * N) want = 2 * N;
    if (want > 65520) want = 65520;
    const size_t base = batch_lds((size_t)N, 0).total + kStaticLds;
    static const size_t tiers[] = {40960, 53248, 81920, 163840};
    int64_t cap = -1;
    for (size_t t : tiers) {
        if (base > t) continue;
        cap = (int64_t)((t - base) & ~(size_t)15);
        if (cap >= want) break;
    }
    if (cap < 2 * N) return s;
    if (cap > 65520) cap = 65520;
    s.cap_n = (int32_t)N;
    s.cap_pairs = (int32_t)cap;
    s.lds_bytes = batch_lds((size_t)N, (size_t)cap).total;
    s.block = N <= (int64_t)kBatchBlock * kMaxItems ? kBatchBlock : kBatchBlockLong;
    int items = 1;  // tensor slots per thread
    while ((int64_t)items * s.block < N) items <<= 1;
    s.items = items;
    s.ok = true;
    return s;
}

size_t plan_batch_workspace_bytes(int64_t n_tensors, int64_t n_traces) {
    if (n_tensors < 0 || n_traces < 0) return 0;
    return (size_t)(kWsPerTensor * n_tensors + kWsPerTrace * n_traces + 64);
}

hipError_t launch_plan_batch(const BatchArgs& a, hipStream_t st) {
    const BatchShape s = batch_shape(a.max_trace_len);
    if (!s.ok) return hipErrorInvalidValue;
    const bool best = a.policy == MP_BEST_FIT;
    constexpr int B = kBatchBlock, BL = kBatchBlockLong;
    if (s.block == BL) {  // longer traces: eight slots a thread
        if (s.items != kMaxItems) return hipErrorInvalidValue;
        return best ? launch_items<BL, 8, true>(a, s, st) : launch_items<BL, 8, false>(a, s, st);
    }
    switch (s.items) {
        case 1: return best ? launch_items<B, 1, true>(a, s, st) : launch_items<B, 1, false>(a, s, st);
        case 2: return best ? launch_items<B, 2, true>(a, s, st) : launch_items<B, 2, false>(a, s, st);
        case 4: return best ? launch_items<B, 4, true>(a, s, st) : launch_items<B, 4, false>(a, s, st);
        case 8: return best ? launch_items<B, 8, true>(a, s, st) : launch_items<B, 8, false>(a, s, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mp
