// Batched greedy-by-size planner: one workgroup per trace, the trace held in LDS.
//
// Method (Section 2.3 greedy_by_size, Section 3.2): tensors are ranked by
// (size desc, first asc, id asc) and each is placed at the lowest offset that
// avoids the byte ranges of the already placed tensors whose lifetimes meet
// its own.  Only lifetime-intersecting pairs interact, so the sequential
// greedy equals evaluating each tensor once all of its "predecessors" --
// intersecting tensors of lower rank -- are placed.  The kernel builds the
// predecessor lists in LDS and places tensors in a dataflow schedule whose
// length is the depth of the predecessor DAG, not the tensor count.
//
// Positions q: the trace's tensors ordered by (first, id).  For q < q' the
// pair intersects iff first[q'] <= last[q], so tensor q meets exactly the
// positions (q, reach[q]) ahead of it, reach[q] = upper_bound(first, last[q]).
// For such a pair q ranks before q' iff size[q] >= size[q'] (equal sizes are
// ordered by first then id, which is position order).
//
// Phases (one workgroup of 512 threads):
//   ingest + checks -> position order -> reach, band prefix, live-bytes deltas
//   -> pair count (balanced over pairs) -> list starts -> list fill ->
//   placement (dataflow: a tensor is fitted once its predecessors are placed)
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
#define MP_STAMP(slot) \
    do {               \
    } while (0)
#define MP_DBG_MAX(slot, v) do { } while (0)
#define MP_DBG_ADD(slot, v) do { } while (0)
#endif
#ifdef MP_PHASE_TIMING
#define MP_CLK(v) long long v = clock64()
#define MP_DBG_CLK_ADD(slot, a, b) \
    do { MP_DBG_ADD(slot, (unsigned)(((b) - (a)) >> 4)); } while (0)
#define MP_DBG_DECL uint32_t dbg_iters = 0, dbg_chunks = 0, dbg_blocks = 0
#define MP_DBG_ITER ++dbg_iters
#define MP_DBG_CHUNK ++dbg_chunks
#define MP_DBG_BLOCK ++dbg_blocks
#define MP_DBG_FLUSH                  \
    do {                              \
        MP_DBG_MAX(0, dbg_iters);     \
        MP_DBG_ADD(1, dbg_iters);     \
        MP_DBG_ADD(2, dbg_chunks);    \
        MP_DBG_ADD(4, dbg_blocks);    \
    } while (0)
#else
#define MP_CLK(v) do { } while (0)
#define MP_DBG_CLK_ADD(slot, a, b) do { } while (0)
#define MP_DBG_DECL do { } while (0)
#define MP_DBG_ITER do { } while (0)
#define MP_DBG_CHUNK do { } while (0)
#define MP_DBG_BLOCK do { } while (0)
#define MP_DBG_FLUSH do { } while (0)
#endif

namespace {

constexpr int kBatchBlock = 512;
constexpr int kChunk = 8;                  // predecessors gathered per round trip
constexpr int kCoopSlots = 4;              // whole-wave fits take up to 4 x 64 predecessors
constexpr uint32_t kCoopMax = 64u * kCoopSlots;

__device__ __forceinline__ uint64_t lds_poll64(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_publish64(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// A tensor's LDS word: offset (units) in the high half, size (units) in the
// low half; the offset half is kUnplaced until the tensor is placed.
__device__ __forceinline__ uint32_t word_off(uint64_t w) { return (uint32_t)(w >> 32); }
__device__ __forceinline__ uint32_t word_end(uint64_t w) {
    return (uint32_t)(w >> 32) + (uint32_t)w;
}

// Gather up to kChunk predecessor ranges [o, e) starting at list index c.
// Slots past `end` read the tensor's own word (`self`) and get an empty
// range that never blocks; the loads are issued unconditionally so that
// they overlap.  Returns the slot of the first predecessor not placed yet,
// or kChunk if all are placed.
__device__ __forceinline__ int gather(const uint16_t* preds, uint32_t c, uint32_t end,
                                      uint32_t self, const uint64_t* ofsz,
                                      uint32_t (&o)[kChunk], uint32_t (&e)[kChunk]) {
    uint32_t idx[kChunk];
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
        const uint32_t v = preds[c + j];  // in bounds: the list area is padded
        idx[j] = (c + j < end) ? v : self;
    }
    uint64_t w[kChunk];
#pragma unroll
    for (int j = 0; j < kChunk; ++j) w[j] = lds_poll64(ofsz + idx[j]);
    int blocked = kChunk;
#pragma unroll
    for (int j = kChunk - 1; j >= 0; --j) {
        const bool live = c + j < end;
        o[j] = live ? word_off(w[j]) : kUnplaced;
        e[j] = live ? word_end(w[j]) : 0u;
        if (live && o[j] == kUnplaced) blocked = j;
    }
    return blocked;
}

// Move x past every range in the chunk that overlaps [x, x + s); any offset
// jumped over overlaps that range, so none of them can fit.  Returns true if
// x moved.
__device__ __forceinline__ bool bump(uint32_t& x, uint32_t s, const uint32_t (&o)[kChunk],
                                     const uint32_t (&e)[kChunk]) {
    bool moved = false;
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
        if (o[j] < x + s && x < e[j]) {
            x = e[j];
            moved = true;
        }
    }
    return moved;
}

// Maximum over the 64 lanes, returned to every lane: DPP row shifts build
// row-wise prefix maxima, row broadcasts carry them across rows, lane 63
// ends up with the total.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false));
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
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

// Exclusive scan of a[0..n) in place (contiguous chunk per thread); a[n] =
// total.  Returns the total.  Barriers inside.
template <int BLOCK>
__device__ uint32_t scan_exclusive_inplace(uint32_t* a, int n, uint32_t* scratch) {
    const int chunk = (n + BLOCK - 1) / BLOCK;
    const int a0 = min(n, (int)threadIdx.x * chunk), a1 = min(n, a0 + chunk);
    uint32_t s = 0;
    for (int i = a0; i < a1; ++i) s += a[i];
    uint32_t total;
    uint32_t run = block_exclusive_sum<BLOCK>(s, &total, scratch);
    for (int i = a0; i < a1; ++i) {
        const uint32_t v = a[i];
        a[i] = run;
        run += v;
    }
    if (threadIdx.x == 0) a[n] = total;
    __syncthreads();
    return total;
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

    // LDS layout (N = cap_n tensor slots, P = cap_pairs list slots):
    //   R0 [8N]     first[N]                     -> placement words ofsz[N]
    //   R1 [4N]     size / unit
    //   R2 [4N+4]   band lengths -> band starts (prefix)
    //   R3 [4N+4]   live-bytes deltas -> predecessor counts -> fill cursors
    //   R4 [4N+4]   predecessor list starts
    //   R5 [2P]     predecessor lists (positions, u16)
    //   R4+R5 hold the u64 sort keys of an unsorted trace before the lists.
    const size_t N = (size_t)cap_n;
    int32_t* fst = reinterpret_cast<int32_t*>(smem);
    uint64_t* ofsz = reinterpret_cast<uint64_t*>(smem);
    uint32_t* sz = reinterpret_cast<uint32_t*>(smem + 8 * N);
    uint32_t* bstart = reinterpret_cast<uint32_t*>(smem + 12 * N);
    uint32_t* cnt = reinterpret_cast<uint32_t*>(smem + 16 * N + 4);
    uint32_t* pbeg = reinterpret_cast<uint32_t*>(smem + 20 * N + 8);
    uint16_t* preds = reinterpret_cast<uint16_t*>(smem + 24 * N + 12);
    uint64_t* keys = reinterpret_cast<uint64_t*>(smem + ((20 * N + 8 + 7) & ~(size_t)7));
    uint32_t* scratch = reinterpret_cast<uint32_t*>(red);

    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    MP_STAMP(0);
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
            sz[q] = su_r[k];
            fst[q] = f_r[k];
            cnt[q] = 0;
        }
    }
    if (tid == 0) cnt[n] = 0;
    __syncthreads();
    MP_STAMP(2);

    // ---- reach (galloping search), band lengths, live-bytes deltas
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
            bstart[q] = (uint32_t)(a - q - 1);
            atomicAdd(&cnt[q], su_r[k]);
            atomicAdd(&cnt[a], 0u - su_r[k]);
        }
    }
    __syncthreads();

    // ---- prefix sums: band starts, max live bytes
    const uint32_t n_band = scan_exclusive_inplace<BLOCK>(bstart, n, scratch);
    uint32_t live_max;
    {
        const int chunk = (n + BLOCK - 1) / BLOCK;
        const int a0 = min(n, tid * chunk), a1 = min(n, a0 + chunk);
        uint32_t ds = 0;
        for (int i = a0; i < a1; ++i) ds += cnt[i];
        uint32_t dtot;
        uint32_t run = block_exclusive_sum<BLOCK>(ds, &dtot, scratch);
        uint32_t lm = 0;
        for (int i = a0; i < a1; ++i) {
            run += cnt[i];
            lm = lm > run ? lm : run;
        }
        live_max = block_reduce<BLOCK>(lm, OpMax<uint32_t>(), scratch);
    }
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        if (q < n) cnt[q] = 0;
    }
    __syncthreads();
    MP_STAMP(3);

    // ---- predecessor counts, balanced over the pairs: pair index p -> (q, j)
    const uint32_t per = (n_band + BLOCK - 1) / BLOCK;
    const uint32_t p_lo = min(n_band, (uint32_t)tid * per), p_hi = min(n_band, p_lo + per);
    int q_lo = 0;  // last position whose band starts at or before p_lo
    if (p_lo < p_hi) {
        int a = 0, z = n;
        while (a < z) {
            const int mid = (a + z + 1) >> 1;
            if (bstart[mid] <= p_lo) a = mid;
            else z = mid - 1;
        }
        q_lo = a;
    }
    if (p_lo < p_hi) {
        int q = q_lo;
        uint32_t nxt = bstart[q + 1];
        uint32_t sq = sz[q];
        for (uint32_t p = p_lo; p < p_hi; ++p) {
            while (nxt <= p) {
                ++q;
                nxt = bstart[q + 1];
                sq = sz[q];
            }
            const int j = q + 1 + (int)(p - bstart[q]);
            const int succ = (sq >= sz[j]) ? j : q;
            atomicAdd(&cnt[succ], 1u);
        }
    }
    __syncthreads();
    const uint32_t n_pairs = scan_exclusive_inplace<BLOCK>(cnt, n, scratch);
    if (n_pairs > (uint32_t)cap_pairs) {
        if (tid == 0) raise_status(status, MP_ENOSPC);
        return;
    }
    for (int i = tid; i <= n; i += BLOCK) pbeg[i] = cnt[i];
    __syncthreads();
    MP_STAMP(4);

    // ---- predecessor lists
    if (p_lo < p_hi) {
        int q = q_lo;
        uint32_t nxt = bstart[q + 1];
        uint32_t sq = sz[q];
        for (uint32_t p = p_lo; p < p_hi; ++p) {
            while (nxt <= p) {
                ++q;
                nxt = bstart[q + 1];
                sq = sz[q];
            }
            const int j = q + 1 + (int)(p - bstart[q]);
            if (sq >= sz[j]) preds[atomicAdd(&cnt[j], 1u)] = (uint16_t)q;
            else preds[atomicAdd(&cnt[q], 1u)] = (uint16_t)j;
        }
    }
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
        const int q = tid + k * BLOCK;
        if (q < n) ofsz[q] = ((uint64_t)kUnplaced << 32) | su_r[k];
    }
    __syncthreads();
    MP_STAMP(5);

    // ---- placement in rounds.  A tensor can be placed once its predecessors
    // are.  Round: (A) every thread looks at the tensors it owns (positions
    // tid + k * BLOCK) that are not placed: a tensor whose remembered blocker
    // is now placed (or that has none) is appended to a ready list -- short
    // predecessor lists to one list, long ones to another; (B) the short
    // ready tensors are spread one per thread: gather the predecessor words,
    // remember the first unplaced one as the new blocker, or fit and publish;
    // the long ready tensors are taken one per wave and handled by the whole
    // wave.  Waves without work wait at the barrier instead of spinning.
    // Every round places at least the lowest-ranked unplaced tensor.
    {
        uint16_t* waitp = reinterpret_cast<uint16_t*>(smem + 8 * N);       // R1
        uint16_t* rsmall = reinterpret_cast<uint16_t*>(smem + 10 * N);     // R1
        uint16_t* rbig = reinterpret_cast<uint16_t*>(smem + 12 * N);       // R2
        uint32_t* cursor = reinterpret_cast<uint32_t*>(smem + 16 * N + 4);  // R3
        __shared__ uint32_t n_small[2], n_big[2], n_placed;
        constexpr uint16_t kNone = 0xFFFF;
        uint32_t todo = 0;
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int q = tid + k * BLOCK;
            if (q < n) {
                todo |= 1u << k;
                waitp[q] = kNone;
                cursor[q] = pbeg[q];
            }
        }
        if (tid == 0) {
            n_small[0] = n_big[0] = n_small[1] = n_big[1] = 0;
            n_placed = 0;
        }
        __syncthreads();
        const int lane = tid & (kWave - 1), wid = tid / kWave;
        constexpr int kWaves = BLOCK / kWave;
        for (int round = 0;; ++round) {
            const int par = round & 1;
            MP_CLK(c0);
            // (A) submit owned tensors whose blocker is gone
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                if (!(todo >> k & 1u)) continue;
                const uint32_t q = tid + k * BLOCK;
                if (word_off(lds_poll64(ofsz + q)) != kUnplaced) {
                    todo &= ~(1u << k);
                    continue;
                }
                const uint16_t w = waitp[q];
                if (w != kNone && word_off(lds_poll64(ofsz + w)) == kUnplaced) continue;
                const uint32_t kp = pbeg[q + 1] - pbeg[q];
                if (kp > (uint32_t)kChunk && kp <= kCoopMax)
                    rbig[atomicAdd(&n_big[par], 1u)] = (uint16_t)q;
                else
                    rsmall[atomicAdd(&n_small[par], 1u)] = (uint16_t)q;
            }
            MP_CLK(c1);
            __syncthreads();
            MP_CLK(c2);
            const uint32_t ns = n_small[par], nb = n_big[par];
            const uint32_t placed_before = n_placed;
            if (tid == 0) n_small[par ^ 1] = n_big[par ^ 1] = 0;
            if (tid == 0) {
                MP_DBG_ADD(1, ns);
                MP_DBG_ADD(2, nb);
            }
            if (placed_before >= (uint32_t)n) {
                if (tid == 0) MP_DBG_MAX(0, round);
                break;
            }
            if (round > n + 2) {  // cannot happen: every round places a tensor
                if (tid == 0) raise_status(status, MP_EDEVICE);
                break;
            }
            // (B1) short lists (and very long ones, chunk by chunk), one per thread
            uint32_t mine = 0;
            for (uint32_t i = tid; i < ns; i += BLOCK) {
                const uint32_t q = rsmall[i];
                const uint32_t pb = pbeg[q], pe = pbeg[q + 1];
                const uint32_t s = (uint32_t)ofsz[q];
                uint32_t o[kChunk], e[kChunk];
                if (pe - pb <= (uint32_t)kChunk) {
                    const int bl = gather(preds, pb, pe, q, ofsz, o, e);
                    if (bl < kChunk) {
                        // wait on the smallest unplaced predecessor: it ranks
                        // last among them, so it is likely placed last
                        int pick = bl;
                        uint32_t best = e[bl] - o[bl];
#pragma unroll
                        for (int j = 0; j < kChunk; ++j) {
                            const uint32_t sj = e[j] - o[j];
                            if (pb + j < pe && o[j] == kUnplaced && sj <= best) {
                                best = sj;
                                pick = j;
                            }
                        }
                        waitp[q] = preds[pb + pick];
                        continue;
                    }
                    uint32_t x = 0;
                    while (bump(x, s, o, e)) {
                    }
                    lds_publish64(ofsz + q, ((uint64_t)x << 32) | s);
                    ++mine;
                    continue;
                }
                uint32_t c = cursor[q];  // very long list: resume the scan
                bool blocked = false;
                while (c < pe) {
                    const int bl = gather(preds, c, pe, q, ofsz, o, e);
                    if (bl < kChunk) {
                        waitp[q] = preds[c + bl];
                        cursor[q] = c + bl;
                        blocked = true;
                        break;
                    }
                    c += kChunk;
                }
                if (blocked) continue;
                const uint32_t nch = (pe - pb + kChunk - 1) / kChunk;
                uint32_t x = 0, cc = pb, clean = 0;
                while (clean < nch) {  // sweep the chunks until a full lap leaves x alone
                    gather(preds, cc, pe, q, ofsz, o, e);
                    bool moved = false;
                    while (bump(x, s, o, e)) moved = true;
                    clean = moved ? 1u : clean + 1u;
                    cc += kChunk;
                    if (cc >= pe) cc = pb;
                }
                lds_publish64(ofsz + q, ((uint64_t)x << 32) | s);
                ++mine;
            }
            MP_CLK(c3);
            // (B2) long lists: one tensor per wave, one predecessor per lane
            // taken from the last wave down, since short ones fill the first waves
            for (uint32_t j = wid; j < nb; j += kWaves) {
                const uint32_t q = rbig[nb - 1 - j];
                const uint32_t upb = pbeg[q], upe = pbeg[q + 1];
                const uint32_t us = (uint32_t)ofsz[q];
                const int slots = (int)((upe - upb + kWave - 1) / kWave);
                uint32_t co[kCoopSlots], ce[kCoopSlots];
                uint64_t w[kCoopSlots];
#pragma unroll
                for (int r = 0; r < kCoopSlots; ++r) {
                    const uint32_t pos = upb + r * kWave + lane;
                    if (r < slots) {
                        const uint32_t v = preds[pos < upe ? pos : upb];
                        w[r] = lds_poll64(ofsz + (pos < upe ? v : q));
                    } else {
                        w[r] = 0;
                    }
                }
                // the smallest unplaced predecessor, if any, becomes the blocker
                uint32_t minsz = 0xFFFFFFFFu, minpos = 0xFFFFFFFFu;
#pragma unroll
                for (int r = 0; r < kCoopSlots; ++r) {
                    const uint32_t pos = upb + r * kWave + lane;
                    const bool live = r < slots && pos < upe;
                    co[r] = live ? word_off(w[r]) : kUnplaced;
                    ce[r] = live ? word_end(w[r]) : 0u;
                    if (live && co[r] == kUnplaced && (uint32_t)w[r] <= minsz) {
                        minsz = (uint32_t)w[r];
                        minpos = pos;
                    }
                }
                const uint32_t wmin = ~wave_max_u32(~minsz);
                if (wmin != 0xFFFFFFFFu) {
                    const uint64_t holders = __ballot(minsz == wmin);
                    const uint32_t pos = (uint32_t)__builtin_amdgcn_readlane(
                        (int)minpos, __ffsll((long long)holders) - 1);
                    if (lane == 0) waitp[q] = preds[pos];
                    continue;
                }
                uint32_t x = 0;
                while (true) {  // jump past the highest end overlapping [x, x + s)
                    bool ov = false;
                    uint32_t mx = 0;
#pragma unroll
                    for (int r = 0; r < kCoopSlots; ++r) {
                        if (co[r] < x + us && x < ce[r]) {
                            ov = true;
                            mx = max(mx, ce[r]);
                        }
                    }
                    if (!__ballot(ov)) break;
                    x = wave_max_u32(mx);
                }
                if (lane == 0) {
                    lds_publish64(ofsz + q, ((uint64_t)x << 32) | us);
                    ++mine;
                }
            }
            if (mine) atomicAdd(&n_placed, mine);
            MP_CLK(c4);
            __syncthreads();
            MP_CLK(c5);
            if (tid == 0) {
                MP_DBG_CLK_ADD(3, c0, c1);
                MP_DBG_CLK_ADD(4, c1, c2);
                MP_DBG_CLK_ADD(5, c2, c3);
                MP_DBG_CLK_ADD(6, c4, c5);
            }
            if (tid == 448) MP_DBG_CLK_ADD(7, c3, c4);
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

// LDS bytes per workgroup: 24 per tensor slot + 16 + 2 per pair slot.  Traces
// up to about 2000 tensors get a budget that lets two workgroups share a CU's
// 160 KiB of LDS.  The sort keys (8 bytes per power-of-two slot) must fit in
// the last two regions.
BatchShape batch_shape(int64_t max_trace_len) {
    BatchShape s{};
    if (max_trace_len < 0 || max_trace_len > MP_BATCH_MAX_TRACE_LEN) return s;
    const int64_t cap_n = max_trace_len < 1 ? 1 : max_trace_len;
    const int64_t fixed = 24 * cap_n + 16;
    const int64_t budget = (fixed <= 48 * 1024) ? 78 * 1024 : 156 * 1024;
    int64_t pairs = (budget - fixed - 16) / 2;
    pairs &= ~(int64_t)7;
    int64_t m = 1;
    while (m < cap_n) m <<= 1;
    if (4 * cap_n + 2 * pairs < 8 * m) return s;  // keys would not fit (never for <= 4096)
    s.cap_n = (int32_t)cap_n;
    s.cap_pairs = (int32_t)pairs;
    s.lds_bytes = (size_t)(fixed + 2 * pairs + 16);  // list reads run up to 8 slots past the end
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
