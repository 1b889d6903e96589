// Greedy-by-size planner for one large trace, using the whole device.
//
// Same method as the batched planner (Section 2.3 greedy_by_size, the
// planner of Section 3.2): tensors ranked by (size desc, first asc, id asc),
// each put at the lowest offset clear of the already placed tensors whose
// lifetimes meet its own.  For a single trace of up to millions of tensors
// the work is spread over the device:
//
//   ingest     checks, common power-of-two unit of the sizes, sortedness
//   positions  order by (first, id) -- a radix sort when not already sorted
//   reach      reach[q] = first position after q born after q dies; the pair
//              (q, j), q < j, intersects iff j < reach[q]
//   long list  positions whose band (q, reach[q]) is longer than a threshold
//              chosen from a histogram of band lengths, so that the other
//              tensors meeting t from behind lie in a short window before t
//   rank       stable radix sort by size descending over positions
//   place      persistent kernel: workgroups take ranks in blocks of 32
//              consecutive ranks claimed per XCD, so that most dependency
//              links (usually rank r - 1 to rank r) stay inside one L2.  For
//              tensor t the workgroup walks t's candidates (forward band,
//              backward window, long list), keeps those ranked before t,
//              turns the already placed ones into one run of ranges by
//              offset (their union through a coverage bitmap, or an LDS
//              bitonic sort with prefix maxima of the ends), marks the run's
//              gaps that hold t, then waits for the rest while keeping the
//              lowest fit up to date as they arrive.  A tensor only waits on
//              lower ranks; each is held by a running workgroup or sits in a
//              block whose XCD takes it once a running workgroup there
//              finishes, so the schedule cannot deadlock.
//   output     offsets (scaled back to bytes) and the peak.
#include <type_traits>
#ifdef MP_DEBUG_WAIT
#include <stdlib.h>
#include <string.h>
#endif

#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr int kTBlock = 512;
constexpr int kRunCap = 16384;    // ranges sorted at once in LDS
// Predecessors still unplaced when t is examined.  Each is held by another
// running workgroup (one rank at a time per workgroup) or is still untaken in
// another XCD's current block (see kTicketBlock), so there are fewer than the
// grid + kXcdGroups * (kTicketBlock - 1); the host keeps the grid at most
// kDynCap + 1 - kXcdGroups * (kTicketBlock - 1).
constexpr int kDynCap = 512;
static_assert(kDynCap <= 8 * kWave, "wave 0 holds every late predecessor, 8 a lane at most");
// Ranks are handed out in blocks of kTicketBlock consecutive ranks: a
// workgroup takes the next slot of its XCD's current block, and the one that
// opens a block claims the next block of the whole trace.  A rank below t's
// can then still be untaken, but only in another XCD's current block (at
// most kTicketBlock - 1 of them per XCD).
constexpr int kXcdGroups = 8;
constexpr uint32_t kTicketBlock = 32;
constexpr uint32_t kUnionMin = 256;  // placed predecessors merged through a bitmap beyond this
constexpr int64_t kScratchRuns = 8;  // global scratch per workgroup: 8 sorted runs
constexpr uint32_t kUnplacedT = 0xFFFFFFFFu;
constexpr int kLongMax = 4096;    // the long list is kept at most this long when possible

constexpr int kPoolSlots = 2;        // shared scratch for predecessor sets beyond a workgroup's own
constexpr uint64_t kUnplaced64 = ~0ull;

struct TFlags {
    uint32_t unsorted, sorted, abort, wide;
    uint64_t or_all, sum;
    uint32_t shift, lthr, n_long, ticket;
    uint32_t xtick[kXcdGroups];  // slots taken per XCD (blocks of kTicketBlock ranks)
    uint32_t blocks;             // rank blocks claimed
    // workgroups finished in ingest, reach and output (the last one of each
    // takes the step that needs all of them)
    uint32_t done_ingest, done_reach, done_output;
    uint32_t skip_narrow, skip_wide;  // nonzero: the 32-bit (64-bit) unit path does not run
    uint32_t pool[kPoolSlots];        // 1 while a workgroup holds the slot
    uint32_t hist[64];      // band lengths by bit width
    uint64_t peak;
    int64_t long_prefix_tiles;
};

struct TView {  // position-ordered arrays
    const int32_t* first;
    const int32_t* last;
    const uint32_t* id;  // null when the input was sorted
};

// ---------------------------------------------------------------- ingest

__global__ void t_init_kernel(TFlags* fl) {
    const int i = threadIdx.x;
    if (i < 64) fl->hist[i] = 0;
    if (i < kPoolSlots) fl->pool[i] = 0;
    if (i < kXcdGroups) fl->xtick[i] = 0;
    if (i == 0) {
        fl->unsorted = 0;
        fl->sorted = 1;
        fl->abort = 0;
        fl->wide = 0;
        fl->skip_narrow = 1;
        fl->skip_wide = 1;
        fl->or_all = 0;
        fl->sum = 0;
        fl->shift = 0;
        fl->lthr = 0;
        fl->n_long = 0;
        fl->ticket = 0;
        fl->blocks = 0;
        fl->done_ingest = 0;
        fl->done_reach = 0;
        fl->done_output = 0;
        fl->peak = 0;
    }
}

__device__ __forceinline__ uint32_t flag_load(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t flag_load64(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Unit shift, and the offset width: 32-bit counts of the unit while the
// sizes sum to less than 2^32 - 1 units (every offset and end then fits
// below the unplaced sentinel), 64-bit counts beyond.  Taken by the last
// ingest workgroup, once every workgroup's totals are in.
__device__ void unit_step(TFlags* fl) {
    if (flag_load(&fl->abort)) return;
    const uint64_t o = flag_load64(&fl->or_all);
    const uint32_t sh = o ? (uint32_t)__builtin_ctzll(o) : 0u;
    fl->shift = sh;
    const uint32_t wide = (flag_load64(&fl->sum) >> sh) > 0xFFFFFFFEull ? 1u : 0u;
    fl->wide = wide;
    fl->skip_narrow = wide;
    fl->skip_wide = 1u - wide;
}

// Checks and totals of the input; besides, the (first, id) pairs of the
// position sort (used only when the input is not sorted by first) and the
// zeroed rank-block table of the placement.
__global__ __launch_bounds__(256) void t_ingest_kernel(const int64_t* __restrict__ size,
                                                       const int32_t* __restrict__ first,
                                                       const int32_t* __restrict__ last,
                                                       int64_t n, int32_t num_ops, TFlags* fl,
                                                       int32_t* __restrict__ status,
                                                       uint64_t* __restrict__ keys,
                                                       uint32_t* __restrict__ vals,
                                                       uint32_t* __restrict__ xbase, int64_t nx) {
    __shared__ uint64_t red[256 / kWave];
    __shared__ uint32_t s_last;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    uint32_t bad = 0, unsorted = 0;
    uint64_t orv = 0, acc = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int64_t s = size[i];
        const int32_t f = first[i], l = last[i];
        if (s <= 0 || f < 0 || f > l || l >= num_ops) bad = 1;
        if (s > 0) {
            orv |= (uint64_t)s;
            acc = sat_add(acc, (uint64_t)s);
        }
        if (i + 1 < n && first[i + 1] < f) unsorted = 1;
        keys[i] = (uint64_t)(uint32_t)f;
        vals[i] = (uint32_t)i;
    }
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nx; i += stride)
        xbase[i] = 0;
    bad = block_reduce<256>(bad, OpOr<uint32_t>(), reinterpret_cast<uint32_t*>(red));
    unsorted = block_reduce<256>(unsorted, OpOr<uint32_t>(), reinterpret_cast<uint32_t*>(red));
    orv = block_reduce<256>(orv, OpOr<uint64_t>(), red);
    acc = block_reduce<256>(acc, OpSatAdd(), red);
    if (threadIdx.x == 0) {
        if (bad) {
            raise_status(status, MP_EINVAL);
            atomicOr(&fl->abort, 1u);
        }
        if (unsorted) {
            atomicOr(&fl->unsorted, 1u);
            atomicAnd(&fl->sorted, 0u);
        }
        atomicOr(reinterpret_cast<unsigned long long*>(&fl->or_all), (unsigned long long)orv);
        const uint64_t old = atomicAdd(reinterpret_cast<unsigned long long*>(&fl->sum),
                                       (unsigned long long)acc);
        if (acc > (uint64_t)INT64_MAX || old > (uint64_t)INT64_MAX - acc) {
            raise_status(status, MP_EOVERFLOW);
            atomicOr(&fl->abort, 1u);
        }
        __threadfence();
        s_last = atomicAdd(&fl->done_ingest, 1u) == gridDim.x - 1 ? 1u : 0u;
    }
    __syncthreads();
    if (s_last && threadIdx.x == 0) {
        __threadfence();
        unit_step(fl);
    }
}

// positions: size in units, first/last in (first, id) order, ids; and the
// rank-sort pairs (size descending; ties keep position order, the sort being
// stable).  perm may be vals (the position sort's result): each thread reads
// its own entry before writing it.
__global__ void t_positions_kernel(const uint32_t* perm,
                                   const int64_t* __restrict__ size,
                                   const int32_t* __restrict__ first,
                                   const int32_t* __restrict__ last, int64_t n,
                                   uint32_t* __restrict__ su, int32_t* __restrict__ pf,
                                   int32_t* __restrict__ pl, uint32_t* __restrict__ pid,
                                   uint32_t* __restrict__ off, uint64_t* __restrict__ su64,
                                   uint64_t* __restrict__ off64, uint64_t* __restrict__ keys,
                                   uint32_t* vals, const TFlags* fl) {
    if (fl->abort) return;
    const bool uns = fl->unsorted != 0, wide = fl->wide != 0;
    const uint32_t sh = fl->shift;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n; q += stride) {
        const uint32_t i = uns ? perm[q] : (uint32_t)q;
        const uint64_t units = (uint64_t)size[i] >> sh;
        if (wide) {
            su64[q] = units;
            off64[q] = kUnplaced64;
            keys[q] = ~units;
        } else {
            su[q] = (uint32_t)units;
            off[q] = kUnplacedT;
            keys[q] = (uint64_t)(0xFFFFFFFFu - (uint32_t)units);
        }
        vals[q] = (uint32_t)q;
        if (uns) {
            pf[q] = first[i];
            pl[q] = last[i];
        }
        pid[q] = i;
    }
}

__device__ __forceinline__ TView view(const TFlags* fl, const int32_t* first, const int32_t* last,
                                      const int32_t* pf, const int32_t* pl, const uint32_t* pid) {
    if (fl->unsorted) return TView{pf, pl, pid};
    return TView{first, last, nullptr};
}

__device__ __forceinline__ int32_t gallop_reach(const int32_t* f, int32_t q, int32_t n,
                                                int32_t l) {
    int64_t known = q, step = 1, probe = (int64_t)q + 1;
    while (probe < n && f[probe] <= l) {
        known = probe;
        step <<= 1;
        probe = ((int64_t)q + step < n) ? (int64_t)q + step : (int64_t)n;
    }
    int64_t a = known + 1, z = probe < n ? probe : (int64_t)n;
    while (a < z) {
        const int64_t mid = a + ((z - a) >> 1);
        if (f[mid] <= l) a = mid + 1;
        else z = mid;
    }
    return (int32_t)a;
}

__global__ void t_reach_kernel(const int32_t* first, const int32_t* last, const int32_t* pf,
                               const int32_t* pl, const uint32_t* pid, int64_t n,
                               int32_t* __restrict__ reach, TFlags* fl) {
    // band-length histogram by bit width: per workgroup in LDS, then one
    // device atomic per nonzero bin (one per position would serialize on the
    // few bins most bands fall in)
    __shared__ uint32_t h[33];
    __shared__ uint32_t s_last;
    if (fl->abort) return;
    if (threadIdx.x < 33) h[threadIdx.x] = 0u;
    __syncthreads();
    const TView v = view(fl, first, last, pf, pl, pid);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n; q += stride) {
        const int32_t r = gallop_reach(v.first, (int32_t)q, (int32_t)n, v.last[q]);
        reach[q] = r;
        const uint32_t band = (uint32_t)(r - q - 1);
        atomicAdd(&h[band ? 32 - __builtin_clz(band) : 0], 1u);
    }
    __syncthreads();
    if (threadIdx.x < 33 && h[threadIdx.x]) atomicAdd(&fl->hist[threadIdx.x], h[threadIdx.x]);
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) s_last = atomicAdd(&fl->done_reach, 1u) == gridDim.x - 1 ? 1u : 0u;
    __syncthreads();
    if (s_last && threadIdx.x == 0) {
        // the last workgroup, all histograms in: the threshold is the
        // smallest 2^b with at most kLongMax bands longer than it
        __threadfence();
        uint32_t above = 0;
        int b = 33;
        // bands of bit width w lie in [2^(w-1), 2^w); count from the top down
        for (int w = 32; w >= 0; --w) {
            const uint32_t c = flag_load(&fl->hist[w]);
            if (above + c > (uint32_t)kLongMax) break;
            above += c;
            b = w;
        }
        // bands with bit width >= b are long: band >= 2^(b-1)
        fl->lthr = (b >= 33) ? 0xFFFFFFFFu : (b <= 1 ? 0u : (1u << (b - 1)) - 1u);
    }
}

__global__ void t_long_flags_kernel(const int32_t* __restrict__ reach, int64_t n,
                                    int64_t* __restrict__ flag, const TFlags* fl) {
    if (fl->abort) return;
    const uint32_t lthr = fl->lthr;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n; q += stride)
        flag[q] = ((uint32_t)(reach[q] - q - 1) > lthr) ? 1 : 0;
}

__global__ void t_long_list_kernel(const int32_t* __restrict__ reach,
                                   const int64_t* __restrict__ pos, int64_t n,
                                   int32_t* __restrict__ long_list, TFlags* fl) {
    if (fl->abort) return;
    const uint32_t lthr = fl->lthr;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n; q += stride) {
        if ((uint32_t)(reach[q] - q - 1) > lthr) long_list[pos[q]] = (int32_t)q;
        if (q == n - 1) fl->n_long = (uint32_t)(pos[q] + (((uint32_t)(reach[q] - q - 1) > lthr) ? 1 : 0));
    }
}

// ---------------------------------------------------------------- placement

// Offsets are published once and carry no other data, so device-coherent
// relaxed accesses suffice (no acquire/release cache maintenance per load).
__device__ __forceinline__ uint32_t agent_load(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// The publish must stay an ordinary (cached) relaxed agent-scope store: a
// non-temporal store was tried and pollers on other XCDs never saw it, so a
// run waiting on such a publish does not end.
__device__ __forceinline__ void agent_store(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t agent_load64(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void agent_store64(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// The next rank for the calling workgroup (thread 0 only): slot c of its
// XCD's counter lies in that XCD's block c / kTicketBlock; the workgroup
// taking slot 0 claims the trace's next block and records it (as block + 1)
// in xbase[x][c / kTicketBlock], where the others of the block read it.
// Blocks are claimed in increasing order and each XCD fills its own in
// order, so every rank is taken once, and a rank below one being placed is
// either held by a running workgroup or waiting in an XCD's current block.
// Any grouping of workgroups would be correct; the XCD is the fast one.
__device__ __forceinline__ uint32_t take_rank(TFlags* fl, uint32_t* xbase, int64_t xcap) {
    uint32_t xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const uint32_t x = xcc & (kXcdGroups - 1);
    const uint32_t c = atomicAdd(&fl->xtick[x], 1u);
    const uint32_t j = c / kTicketBlock, s = c % kTicketBlock;
    uint32_t* slot = xbase + (int64_t)x * xcap + j;
    if (s == 0) {
        const uint32_t blk = atomicAdd(&fl->blocks, 1u);
        agent_store(slot, blk + 1u);
        return blk * kTicketBlock;
    }
    uint32_t v;
    while ((v = agent_load(slot)) == 0u) __builtin_amdgcn_s_sleep(1);
    return (v - 1u) * kTicketBlock + s;
}
// Barrier after which every thread's global stores of the workgroup are
// complete (the workgroup barrier alone does not wait for them); readers then
// load through L2 (agent_load64).
__device__ __forceinline__ void l2_barrier() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
}

template <int BLOCK>
__device__ void bitonic_sort_keys(uint64_t* keys, int m) {
    for (int k = 2; k <= m; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < (m >> 1); i += BLOCK) {
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

// A run: byte ranges as keys (start << 32 | end) sorted ascending; after
// sorting, the low half of key i is replaced by the maximum end of keys
// 0..i.  The start of key i and the prefix maximum below it are all the
// fit needs.
__device__ __forceinline__ uint32_t run_start(uint64_t k) { return (uint32_t)(k >> 32); }
__device__ __forceinline__ uint32_t run_pmax(uint64_t k) { return (uint32_t)k; }

// Sort keys[0..m0) in LDS (padded to a power of two) and turn the low halves
// into prefix maxima of the ends.  Contiguous chunk per thread for the scan.
template <int BLOCK>
__device__ void make_run(uint64_t* keys, int m0, uint32_t* scratch) {
    int m = 1;
    while (m < m0) m <<= 1;
    for (int i = m0 + threadIdx.x; i < m; i += BLOCK) keys[i] = ~0ull;
    __syncthreads();
    bitonic_sort_keys<BLOCK>(keys, m);
    const int chunk = (m0 + BLOCK - 1) / BLOCK;
    const int a0 = min(m0, (int)threadIdx.x * chunk), a1 = min(m0, a0 + chunk);
    uint32_t local = 0;
    for (int i = a0; i < a1; ++i) local = max(local, (uint32_t)keys[i]);
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    uint32_t inc = local;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(inc, o, kWave);
        if (lane >= o) inc = max(inc, y);
    }
    if (lane == kWave - 1) scratch[wid] = inc;
    __syncthreads();
    uint32_t run = 0;
    for (int w = 0; w < wid; ++w) run = max(run, scratch[w]);
    const uint32_t prev_lane = __shfl_up(inc, 1, kWave);
    if (lane > 0) run = max(run, prev_lane);
    for (int i = a0; i < a1; ++i) {
        run = max(run, (uint32_t)keys[i]);
        keys[i] = (keys[i] & 0xFFFFFFFF00000000ull) | run;
    }
    __syncthreads();
}

// Is [c, c + s) clear of every range of the run?  The ranges starting below
// c + s are a prefix of the run; their highest end must not exceed c.
__device__ __forceinline__ bool run_clear(const uint64_t* keys, int m, uint32_t c, uint32_t s) {
    int a = 0, z = m;  // first key with start >= c + s
    const uint32_t lim = c + s;
    while (a < z) {
        const int mid = (a + z) >> 1;
        if (run_start(keys[mid]) < lim) a = mid + 1;
        else z = mid;
    }
    return a == 0 || run_pmax(keys[a - 1]) <= c;
}

// The placed predecessors as one run of disjoint ranges, when their union is
// compact: the union drawn as a coverage bitmap over offset units (in the LDS
// that holds a run), then its maximal covered intervals, in address order,
// written back over the keys as start << 32 | end (disjoint, so each end is
// its own prefix maximum) and loaded into `skeys`.  The lowest and the
// tightest fit depend on the union only.  Returns false, the keys untouched,
// when the union reaches past kRunCap * 64 units or has more than kRunCap
// intervals.
template <int BLOCK>
__device__ bool union_run(uint64_t* gkeys, uint32_t nstat, uint64_t* skeys, uint32_t* scratch,
                          uint64_t* scratch64, uint32_t* m_out) {
    constexpr uint32_t kBits = (uint32_t)kRunCap * 64u;
    uint32_t top = 0;
    for (uint32_t i = threadIdx.x; i < nstat; i += BLOCK) top = max(top, (uint32_t)gkeys[i]);
    top = block_reduce<BLOCK>(top, OpMax<uint32_t>(), scratch);
    if (top > kBits) return false;
    uint32_t* bm = reinterpret_cast<uint32_t*>(skeys);
    const uint32_t nw = (top + 31) >> 5;
    for (uint32_t j = threadIdx.x; j < nw; j += BLOCK) bm[j] = 0u;
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < nstat; i += BLOCK) {
        const uint64_t k = gkeys[i];
        const uint32_t o = (uint32_t)(k >> 32), e = (uint32_t)k;  // e > o
        const uint32_t w0 = o >> 5, w1 = (e - 1) >> 5;
        const uint32_t m0 = 0xFFFFFFFFu << (o & 31), m1 = 0xFFFFFFFFu >> (31 - ((e - 1) & 31));
        if (w0 == w1) {
            atomicOr(&bm[w0], m0 & m1);
        } else {
            atomicOr(&bm[w0], m0);
            // full words: any interleaving with other writers leaves all ones
            for (uint32_t j = w0 + 1; j < w1; ++j) bm[j] = 0xFFFFFFFFu;
            atomicOr(&bm[w1], m1);
        }
    }
    __syncthreads();
    // interval starts (a covered unit after an uncovered one) and ends (the
    // reverse), counted per contiguous chunk of words; the k-th start and the
    // k-th end bound the k-th interval
    const uint32_t chunk = (nw + BLOCK - 1) / BLOCK;
    const uint32_t j0 = min(nw, (uint32_t)threadIdx.x * chunk), j1 = min(nw, j0 + chunk);
    auto edges = [&](uint32_t j, uint32_t& st, uint32_t& en) {
        const uint32_t w = bm[j];
        const uint32_t prev = j ? bm[j - 1] >> 31 : 0u;
        const uint32_t next = j + 1 < nw ? bm[j + 1] & 1u : 0u;
        st = w & ~((w << 1) | prev);
        en = w & ~((w >> 1) | (next << 31));
    };
    uint32_t cs = 0, ce = 0;
    for (uint32_t j = j0; j < j1; ++j) {
        uint32_t st, en;
        edges(j, st, en);
        cs += (uint32_t)__popc(st);
        ce += (uint32_t)__popc(en);
    }
    uint64_t total;
    const uint64_t base =
        block_exclusive_sum<BLOCK, uint64_t>(((uint64_t)cs << 32) | ce, &total, scratch64);
    const uint32_t m = (uint32_t)total;
    if (m > (uint32_t)kRunCap) return false;
    uint32_t* g32 = reinterpret_cast<uint32_t*>(gkeys);  // key k: [2k] end, [2k + 1] start
    uint32_t gs = (uint32_t)(base >> 32), ge = (uint32_t)base;
    for (uint32_t j = j0; j < j1; ++j) {
        uint32_t st, en;
        edges(j, st, en);
        for (; st; st &= st - 1) g32[2 * gs++ + 1] = 32u * j + (uint32_t)__builtin_ctz(st);
        for (; en; en &= en - 1) g32[2 * ge++] = 32u * j + (uint32_t)__builtin_ctz(en) + 1u;
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < m; i += BLOCK) skeys[i] = gkeys[i];
    __syncthreads();
    *m_out = m;
    return true;
}

// Lowest offset clear of every run.  It is 0 or the end of some range; an
// end that is clear of its own run is the prefix maximum just below a gap of
// at least s in that run (or the run's top), so those gap starts, checked
// against the other runs, are the only candidates.
struct RunRef {
    const uint64_t* keys;
    int m;
};

template <int BLOCK, int MAXR>
__device__ uint32_t fit_runs(const RunRef (&runs)[MAXR], int nr, uint32_t s, uint32_t* scratch) {
    uint32_t best = 0xFFFFFFFFu;
    for (int r = 0; r < nr; ++r) {
        const uint64_t* k = runs[r].keys;
        const int m = runs[r].m;
        for (int i = threadIdx.x; i <= m; i += BLOCK) {
            const uint32_t c = (i == 0) ? 0u : run_pmax(k[i - 1]);
            if (c >= best) continue;
            if (i < m && run_start(k[i]) < c + s) continue;  // no room in this run
            bool ok = true;
            for (int r2 = 0; r2 < nr && ok; ++r2)
                if (r2 != r) ok = run_clear(runs[r2].keys, runs[r2].m, c, s);
            if (ok) best = c;
        }
    }
    return block_reduce<BLOCK>(best, OpMin<uint32_t>(), scratch);
}

// BEST_FIT over the union of the runs (the tightest-gap reading of Section
// 2.3's "best fit"): the smallest free gap that holds s wins, the lowest
// start among equals, and the top of the union only when no gap holds s.  A
// free gap of the union starts at 0 or at the prefix maximum below some key
// (or at the top) of one run, at a point no other run covers, and reaches the
// lowest start at or above that point in any run.
template <int BLOCK, int MAXR>
__device__ uint32_t best_fit_runs(const RunRef (&runs)[MAXR], int nr, uint32_t s,
                                  uint64_t* scratch) {
    uint64_t best = ~0ull;
    uint32_t top = 0;
    for (int r = 0; r < nr; ++r) {
        const uint64_t* k = runs[r].keys;
        const int m = runs[r].m;
        if (m == 0) continue;
        top = max(top, run_pmax(k[m - 1]));
        for (int i = threadIdx.x; i <= m; i += BLOCK) {
            const uint32_t c = (i == 0) ? 0u : run_pmax(k[i - 1]);
            uint64_t end = (i < m) ? (uint64_t)run_start(k[i]) : ~0ull;
            if (end < (uint64_t)c + s) continue;  // gap of this run too small
            for (int r2 = 0; r2 < nr && end >= (uint64_t)c + s; ++r2) {
                if (r2 == r) continue;
                const uint64_t* k2 = runs[r2].keys;
                int a = 0, z = runs[r2].m;  // first key with start >= c
                while (a < z) {
                    const int mid = (a + z) >> 1;
                    if (run_start(k2[mid]) < c) a = mid + 1;
                    else z = mid;
                }
                if (a > 0 && run_pmax(k2[a - 1]) > c) end = 0;  // c is covered
                else if (a < runs[r2].m) end = min(end, (uint64_t)run_start(k2[a]));
            }
            if (end == ~0ull || end < (uint64_t)c + s) continue;  // the top, or too small
            const uint64_t key = ((end - c) << 32) | c;
            best = key < best ? key : best;
        }
    }
    best = block_reduce<BLOCK>(best, OpMin<uint64_t>(), scratch);
    return best != ~0ull ? (uint32_t)best : top;
}

struct PlaceArgs {
    const uint32_t* su;
    const int32_t* reach;
    const uint32_t* order;
    const int32_t* long_list;
    uint32_t* off;
    uint64_t* run_keys;  // per workgroup: stat_cap keys
    int64_t stat_cap;    // min(4 n, kScratchRuns * kRunCap)
    uint64_t* pool;      // kPoolSlots x 4 arrays of n ranges, for larger predecessor sets
    int64_t n;
    TFlags* fl;
    int32_t* status;
    // fit policy: 0 lowest gap, 1 tightest gap (a build with MP_DEBUG_WAIT
    // also reads bits 8 and 9: a late list of 8; the widest wait)
    int32_t best;
    uint32_t* xbase;  // kXcdGroups x xcap claimed blocks (+1), zero at the launch
    int64_t xcap;
};

// Visit the positions ranked before t whose lifetimes meet t's: the forward
// band, the backward window of short bands and the long list; fn(p, o) gets
// each with its offset as read (kUnplacedT while not placed).  Each thread
// takes kBatch candidates per turn and issues their loads together (sizes
// and reaches, then offsets), so the latencies overlap.  With 32-bit sizes
// the forward band and the backward window are read 4 kVec positions a
// thread per turn, four consecutive ones per 16-byte load.  A forward band
// longer than one such pass (a long-lived tensor's spans most of the trace,
// and its walk was a chain of dependent turns) goes in two steps per
// segment of kBandSeg positions: its sizes, 4 kBandVec positions a thread
// per turn, filter the candidates into an LDS list (no offset load waits on
// a size load), then the listed candidates' offsets are loaded kBandLoads a
// thread at a time.  Decode-like trace: 52.4 -> 49.7 ms.
constexpr int kBatch = 4;
constexpr int kVec = 4;
constexpr int kBandVec = 8;
constexpr int32_t kBandSeg = 2 * kRunCap;  // list entries (u32) in the run buffer
constexpr int kBandLoads = 8;

// The candidate walk over positions, for either width of sizes (SZ) and
// offsets (OF, kUnplaced of that width while unplaced).
// The 32-bit path passes an LDS list of kBandSeg entries and its counter
// (every thread of the workgroup calls the walk; it holds barriers then).
template <int BLOCK, typename SZ, typename OF, typename F>
__device__ __forceinline__ void walk_preds(const int32_t* reach, const SZ* su, const OF* off,
                                           const int32_t* long_list, int32_t qt, SZ st,
                                           uint32_t lthr, uint32_t n_long, F&& fn,
                                           uint32_t* list = nullptr, uint32_t* list_n = nullptr) {
    auto load_off = [&](int32_t p) -> OF {
        if constexpr (sizeof(OF) == 8) return agent_load64(reinterpret_cast<const uint64_t*>(off) + p);
        else return agent_load(reinterpret_cast<const uint32_t*>(off) + p);
    };
    auto finish = [&](const auto& pp, const auto& ok) {
        constexpr int N = sizeof(pp) / sizeof(pp[0]);
        OF o[N];
#pragma unroll
        for (int u = 0; u < N; ++u) o[u] = ok[u] ? load_off(pp[u]) : OF(0);
#pragma unroll
        for (int u = 0; u < N; ++u)
            if (ok[u]) fn(pp[u], o[u]);
    };
    const int32_t rt = reach[qt];
    const int64_t lo = (int64_t)qt - (int64_t)lthr - 1;
    if constexpr (sizeof(SZ) == 4) {
        // positions g .. g + 3 (g a multiple of 4) below `end`: one 16-byte
        // load when all four are, else one load per position below `end`
        auto load4 = [&](const auto* arr, int32_t g, int32_t end, auto (&v)[4]) {
            using T = std::remove_cv_t<std::remove_reference_t<decltype(arr[0])>>;
            if (g + 3 < end) {
                const uint4 w = *reinterpret_cast<const uint4*>(arr + g);
                v[0] = (T)w.x; v[1] = (T)w.y; v[2] = (T)w.z; v[3] = (T)w.w;
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = g + e < end ? arr[g + e] : T(0);
            }
        };
        constexpr int32_t kStride = 4 * BLOCK;  // positions between a thread's groups
        // forward band: meets t; ranked before t iff strictly larger
        if (rt - qt - 1 <= kStride * kVec) {  // one pass
            for (int32_t g0 = ((qt + 1) & ~3) + 4 * (int32_t)threadIdx.x; g0 < rt;
                 g0 += kStride * kVec) {
                uint32_t sz[kVec][4];
#pragma unroll
                for (int k = 0; k < kVec; ++k) load4(su, g0 + kStride * k, rt, sz[k]);
                int32_t pp[4 * kVec];
                bool ok[4 * kVec];
#pragma unroll
                for (int k = 0; k < kVec; ++k)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int32_t p = g0 + kStride * k + e;
                        pp[4 * k + e] = p;
                        ok[4 * k + e] = p > qt && p < rt && sz[k][e] > st;
                    }
                finish(pp, ok);
            }
        } else {
            for (int32_t s0 = qt + 1; s0 < rt; s0 += kBandSeg) {
                const int32_t s1 = rt - s0 > kBandSeg ? s0 + kBandSeg : rt;
                if (threadIdx.x == 0) *list_n = 0;
                __syncthreads();
                for (int32_t g0 = (s0 & ~3) + 4 * (int32_t)threadIdx.x; g0 < s1;
                     g0 += kStride * kBandVec) {
                    uint32_t sz[kBandVec][4];
    #pragma unroll
                    for (int k = 0; k < kBandVec; ++k) load4(su, g0 + kStride * k, s1, sz[k]);
    #pragma unroll
                    for (int k = 0; k < kBandVec; ++k)
    #pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int32_t p = g0 + kStride * k + e;
                            if (p >= s0 && p < s1 && sz[k][e] > st) list[atomicAdd(list_n, 1u)] = (uint32_t)p;
                        }
                }
                __syncthreads();
                const uint32_t m = *list_n;
                for (uint32_t i0 = threadIdx.x; i0 < m; i0 += BLOCK * kBandLoads) {
                    int32_t pp[kBandLoads];
                    bool ok[kBandLoads];
    #pragma unroll
                    for (int u = 0; u < kBandLoads; ++u) {
                        const uint32_t i = i0 + (uint32_t)(u * BLOCK);
                        ok[u] = i < m;
                        pp[u] = ok[u] ? (int32_t)list[i] : 0;
                    }
                    finish(pp, ok);
                }
                __syncthreads();  // the list is refilled or handed back
            }
        }
        // backward window of short bands: ranked before t iff at least as large
        const int32_t w0 = (int32_t)(lo > 0 ? lo : 0);
        for (int32_t g0 = (w0 & ~3) + 4 * (int32_t)threadIdx.x; g0 < qt; g0 += kStride * kVec) {
            uint32_t sz[kVec][4];
            int32_t rr[kVec][4];
#pragma unroll
            for (int k = 0; k < kVec; ++k) {
                load4(su, g0 + kStride * k, qt, sz[k]);
                load4(reach, g0 + kStride * k, qt, rr[k]);
            }
            int32_t pp[4 * kVec];
            bool ok[4 * kVec];
#pragma unroll
            for (int k = 0; k < kVec; ++k)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int32_t p = g0 + kStride * k + e;
                    pp[4 * k + e] = p;
                    ok[4 * k + e] = p >= w0 && p < qt && (uint32_t)(rr[k][e] - p - 1) <= lthr &&
                                    rr[k][e] > qt && sz[k][e] >= st;
                }
            finish(pp, ok);
        }
    } else {
    // forward band: meets t; ranked before t iff strictly larger
    for (int32_t j0 = qt + 1 + (int32_t)threadIdx.x; j0 < rt; j0 += BLOCK * kBatch) {
        int32_t pp[kBatch];
        bool ok[kBatch];
        SZ sz[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            pp[u] = j0 + u * BLOCK;
            sz[u] = pp[u] < rt ? su[pp[u]] : SZ(0);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) ok[u] = pp[u] < rt && sz[u] > st;
        finish(pp, ok);
    }
    // backward window of short bands: ranked before t iff at least as large
    for (int64_t p0 = (lo > 0 ? lo : 0) + threadIdx.x; p0 < qt; p0 += BLOCK * kBatch) {
        int32_t pp[kBatch], rr[kBatch];
        bool ok[kBatch];
        SZ sz[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int64_t p = p0 + (int64_t)u * BLOCK;
            pp[u] = (int32_t)p;
            rr[u] = p < qt ? reach[p] : 0;
            sz[u] = p < qt ? su[p] : SZ(0);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            ok[u] = pp[u] < qt && (uint32_t)(rr[u] - pp[u] - 1) <= lthr && rr[u] > qt && sz[u] >= st;
        finish(pp, ok);
    }
    }
    // long bands that started before t
    for (uint32_t k0 = threadIdx.x; k0 < n_long; k0 += BLOCK * kBatch) {
        int32_t pp[kBatch], rr[kBatch];
        bool ok[kBatch];
        SZ sz[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const uint32_t k = k0 + u * BLOCK;
            pp[u] = k < n_long ? long_list[k] : qt;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            rr[u] = pp[u] < qt ? reach[pp[u]] : 0;
            sz[u] = pp[u] < qt ? su[pp[u]] : SZ(0);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) ok[u] = pp[u] < qt && rr[u] > qt && sz[u] >= st;
        finish(pp, ok);
    }
}

template <int BLOCK, typename F>
__device__ __forceinline__ void for_each_pred(const PlaceArgs& a, int32_t qt, uint32_t st,
                                              uint32_t lthr, uint32_t n_long, uint32_t* list,
                                              uint32_t* list_n, F&& fn) {
    walk_preds<BLOCK, uint32_t, uint32_t>(a.reach, a.su, a.off, a.long_list, qt, st, lthr,
                                          n_long, fn, list, list_n);
}

// ------------------------------------------------- general fit (any width)
//
// The placed predecessors of a tensor as byte ranges (start, end), 64-bit, in
// two global arrays (ks, ke) with a second pair (ts, te) of the same length
// for merging: sorted by start in LDS runs of kGRun, runs merged pairwise
// (merge path: each thread's share of the output found by a binary search on
// the two runs), then one pass over the sorted ranges with running maxima of
// the ends -- the gap before range i runs from the maximum end below it to
// its start.  Lowest fit: the first gap that holds s, else the top; BEST_FIT:
// the tightest such gap (lowest start among equals), else the top.  Every
// thread returns the offset.  Global reads of data other threads wrote go
// through L2 (agent_load64) after an l2_barrier.
constexpr int kGRun = 8192;

struct GenRanges {
    uint64_t* ks;
    uint64_t* ke;
    uint64_t* ts;
    uint64_t* te;
};

template <int BLOCK>
__device__ uint64_t fit_general(GenRanges g, uint32_t m, uint64_t s, bool best, uint64_t* lks,
                                uint64_t* lke, uint64_t* red64) {
    const int tid = threadIdx.x;
    l2_barrier();
    // 1. runs of kGRun sorted by start in LDS
    for (uint32_t r0 = 0; r0 < m; r0 += kGRun) {
        const uint32_t len = min((uint32_t)kGRun, m - r0);
        uint32_t p2 = 1;
        while (p2 < len) p2 <<= 1;
        for (uint32_t i = tid; i < p2; i += BLOCK) {
            lks[i] = i < len ? agent_load64(g.ks + r0 + i) : ~0ull;
            lke[i] = i < len ? agent_load64(g.ke + r0 + i) : 0ull;
        }
        __syncthreads();
        for (uint32_t k = 2; k <= p2; k <<= 1) {
            for (uint32_t j = k >> 1; j > 0; j >>= 1) {
                for (uint32_t i = tid; i < (p2 >> 1); i += BLOCK) {
                    const uint32_t lo = ((i & ~(j - 1)) << 1) | (i & (j - 1)), hi = lo | j;
                    const uint64_t a = lks[lo], b = lks[hi];
                    const bool up = (lo & k) == 0;
                    if ((a > b) == up) {
                        lks[lo] = b;
                        lks[hi] = a;
                        const uint64_t ea = lke[lo];
                        lke[lo] = lke[hi];
                        lke[hi] = ea;
                    }
                }
                __syncthreads();
            }
        }
        for (uint32_t i = tid; i < len; i += BLOCK) {
            g.ks[r0 + i] = lks[i];
            g.ke[r0 + i] = lke[i];
        }
        __syncthreads();
    }
    // 2. pairwise merges of runs of width w, ping-ponging between the arrays
    for (uint32_t w = kGRun; w < m; w <<= 1) {
        l2_barrier();
        const uint32_t chunk = (m + BLOCK - 1) / BLOCK;
        const uint32_t o0 = min(m, (uint32_t)tid * chunk), o1 = min(m, o0 + chunk);
        for (uint32_t o = o0; o < o1;) {
            const uint32_t base = o / (2 * w) * (2 * w);  // this output's pair of runs
            const uint32_t la = min(w, m - base), lb = min(w, m - base - la);
            const uint64_t* A = g.ks + base;
            const uint64_t* B = g.ks + base + la;
            const uint32_t d = o - base, stop = min(o1, base + la + lb);
            // co-rank: i outputs of the d come from A
            uint32_t lo = d > lb ? d - lb : 0u, hi = min(d, la);
            while (lo < hi) {
                const uint32_t i = (lo + hi) >> 1;
                if (agent_load64(B + (d - i - 1)) < agent_load64(A + i)) hi = i;
                else lo = i + 1;
            }
            uint32_t i = lo, j = d - lo;
            for (; o < stop; ++o) {
                const bool fromA =
                    j >= lb || (i < la && agent_load64(A + i) <= agent_load64(B + j));
                const uint32_t src = fromA ? base + i : base + la + j;
                g.ts[o] = agent_load64(g.ks + src);
                g.te[o] = agent_load64(g.ke + src);
                i += fromA ? 1u : 0u;
                j += fromA ? 0u : 1u;
            }
        }
        uint64_t* t0 = g.ks;
        uint64_t* t1 = g.ke;
        g.ks = g.ts;
        g.ke = g.te;
        g.ts = t0;
        g.te = t1;
    }
    l2_barrier();
    // 3. one pass over the sorted ranges
    const uint32_t chunk = (m + BLOCK - 1) / BLOCK;
    const uint32_t e0 = min(m, (uint32_t)tid * chunk), e1 = min(m, e0 + chunk);
    uint64_t hi_end = 0;
    for (uint32_t e = e0; e < e1; ++e) hi_end = max(hi_end, agent_load64(g.ke + e));
    // running maximum of the ends before this thread's chunk, and overall
    const int lane = tid & (kWave - 1), wid = tid / kWave;
    uint64_t inc = hi_end;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint64_t y = __shfl_up(inc, d, kWave);
        if (lane >= d) inc = max(inc, y);
    }
    if (lane == kWave - 1) red64[wid] = inc;
    __syncthreads();
    uint64_t run = 0, top = 0;
#pragma unroll
    for (int w = 0; w < BLOCK / kWave; ++w) {
        const uint64_t t = red64[w];
        run = w < wid ? max(run, t) : run;
        top = max(top, t);
    }
    __syncthreads();
    uint64_t prev = __shfl_up(inc, 1, kWave);
    run = max(run, lane ? prev : 0ull);
    uint64_t cand = ~0ull, cgap = ~0ull;
    for (uint32_t e = e0; e < e1; ++e) {
        const uint64_t st = agent_load64(g.ks + e), en = agent_load64(g.ke + e);
        if (st >= run && st - run >= s) {
            if (!best) {
                if (cand == ~0ull) cand = run;
            } else if (st - run < cgap) {
                cgap = st - run;
                cand = run;
            }
        }
        run = max(run, en);
    }
    uint64_t x;
    if (!best) {
        x = block_reduce<BLOCK>(cand, OpMin<uint64_t>(), red64);
    } else {
        const uint64_t gm = block_reduce<BLOCK>(cgap, OpMin<uint64_t>(), red64);
        x = block_reduce<BLOCK>(cgap == gm ? cand : ~(uint64_t)0, OpMin<uint64_t>(), red64);
    }
    return x == ~0ull ? top : x;
}

// One of the kPoolSlots shared predecessor buffers (n ranges each), taken
// only by a workgroup whose tensor has all its predecessors placed, so a
// holder never waits on anything and every wait for a slot ends.  Thread 0
// takes it; every thread gets its index.
__device__ uint32_t pool_acquire(TFlags* fl, uint32_t* s_slot) {
    if (threadIdx.x == 0) {
        uint32_t slot = 0;
        while (true) {
            for (slot = 0; slot < (uint32_t)kPoolSlots; ++slot)
                if (atomicCAS(&fl->pool[slot], 0u, 1u) == 0u) break;
            if (slot < (uint32_t)kPoolSlots) break;
            __builtin_amdgcn_s_sleep(16);
        }
        *s_slot = slot;
    }
    __threadfence();
    __syncthreads();
    return *s_slot;
}
__device__ void pool_release(TFlags* fl, uint32_t slot) {
    l2_barrier();
    if (threadIdx.x == 0) {
        __threadfence();
        atomicExch(&fl->pool[slot], 0u);
    }
}
__device__ __forceinline__ GenRanges pool_ranges(uint64_t* pool, uint32_t slot, int64_t n) {
    uint64_t* b = pool + (int64_t)slot * 4 * n;
    return GenRanges{b, b + n, b + 2 * n, b + 3 * n};
}

// Placement with 64-bit unit counts (the sizes sum to 2^32 - 1 units or
// more): the same ticket order, each workgroup waiting for every
// predecessor of its tensor before the general fit; the ranges go to the
// workgroup's own buffers (cap each) or, beyond, to a pool slot.
struct WideArgs {
    const uint64_t* su;
    const int32_t* reach;
    const uint32_t* order;
    const int32_t* long_list;
    uint64_t* off;
    uint64_t* priv;  // per workgroup: 4 arrays of cap ranges
    int64_t cap;
    uint64_t* pool;  // kPoolSlots x 4 arrays of n
    int64_t n;
    TFlags* fl;
    int32_t best;
};

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void t_place_wide_kernel(WideArgs a) {
    __shared__ uint64_t lks[kGRun];
    __shared__ uint64_t lke[kGRun];
    __shared__ uint64_t red64[BLOCK / kWave];
    __shared__ uint32_t s_rank, s_cnt, s_slot;
    if (a.fl->abort || !a.fl->wide) return;
    const uint32_t lthr = a.fl->lthr, n_long = a.fl->n_long;
    uint64_t* pv = a.priv + (int64_t)blockIdx.x * 4 * a.cap;
    const GenRanges own{pv, pv + a.cap, pv + 2 * a.cap, pv + 3 * a.cap};
    while (true) {
        if (threadIdx.x == 0) {
            s_rank = atomicAdd(&a.fl->ticket, 1u);
            s_cnt = 0;
        }
        __syncthreads();
        const uint32_t r = s_rank;
        if (r >= (uint64_t)a.n) break;
        const int32_t qt = (int32_t)a.order[r];
        const uint64_t st = a.su[qt];
        auto collect = [&](const GenRanges& gr, int64_t cap) {
            walk_preds<BLOCK, uint64_t, uint64_t>(
                a.reach, a.su, a.off, a.long_list, qt, st, lthr, n_long, [&](int32_t p, uint64_t o) {
                    while (o == kUnplaced64) {  // a lower rank, held by a running workgroup
                        __builtin_amdgcn_s_sleep(2);
                        o = agent_load64(a.off + p);
                    }
                    const uint32_t k = atomicAdd(&s_cnt, 1u);
                    if (k < cap) {
                        gr.ks[k] = o;
                        gr.ke[k] = o + a.su[p];
                    }
                });
            __syncthreads();
        };
        collect(own, a.cap);
        const uint32_t m = s_cnt;
        uint64_t x;
        if (m <= a.cap) {
            x = fit_general<BLOCK>(own, m, st, a.best != 0, lks, lke, red64);
        } else {  // every predecessor is placed now: a pool slot, the ranges again
            const uint32_t slot = pool_acquire(a.fl, &s_slot);
            const GenRanges gr = pool_ranges(a.pool, slot, a.n);
            __syncthreads();
            if (threadIdx.x == 0) s_cnt = 0;
            __syncthreads();
            collect(gr, a.n);
            x = fit_general<BLOCK>(gr, s_cnt, st, a.best != 0, lks, lke, red64);
            pool_release(a.fl, slot);
        }
        if (threadIdx.x == 0) agent_store64(a.off + qt, x);
        __syncthreads();
    }
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void t_place_kernel(PlaceArgs a) {
#ifdef MP_DEBUG_WAIT
    // test build (MEMOPLAN_DEBUG_WAIT bits of a.best): 0x200 every wait takes
    // its widest form; 0x100 besides the late list holds 8
#define T_DYN_CAP ((a.best & 0x100) ? 8u : (uint32_t)kDynCap)
#define T_BEST (a.best & 1)
#define T_WIDEST_WAIT ((a.best & 0x200) != 0)
#else
#define T_DYN_CAP ((uint32_t)kDynCap)
#define T_BEST a.best
#define T_WIDEST_WAIT false
#endif
    __shared__ uint64_t skeys[kRunCap];  // placed predecessors (one run)
    __shared__ uint64_t dkeys[kDynCap];  // predecessors placed after t was examined
    __shared__ uint32_t dpos[kDynCap];
    __shared__ uint32_t scratch[BLOCK / kWave];
    __shared__ uint64_t scratch64[BLOCK / kWave];
    __shared__ uint64_t gbits[kRunCap / 64];  // gaps of the placed run that hold t
    __shared__ uint32_t cidx[kWave];           // the first 64 of them
    __shared__ uint32_t s_rank, s_nstat, s_ndyn, s_slot, s_lcnt;
    // the run buffer is free while predecessors are collected: the forward
    // band's candidate list
    uint32_t* const band_list = reinterpret_cast<uint32_t*>(skeys);
    if (a.fl->abort || a.fl->wide) return;
    const uint32_t lthr = a.fl->lthr, n_long = a.fl->n_long;
    uint64_t* gkeys = a.run_keys + (int64_t)blockIdx.x * a.stat_cap;
    const int64_t stat_cap = a.stat_cap;
    while (true) {
        if (threadIdx.x == 0) {
            s_rank = take_rank(a.fl, a.xbase, a.xcap);
            s_nstat = 0;
            s_ndyn = 0;
        }
        __syncthreads();
        const uint32_t r = s_rank;
        if (r >= (uint32_t)a.n) break;
        const int32_t qt = (int32_t)a.order[r];
        const uint32_t st = a.su[qt];
        // 1. collect: placed predecessors as keys, unplaced ones by position
        //    (beyond kDynCap of those, wait for them right here)
        for_each_pred<BLOCK>(a, qt, st, lthr, n_long, band_list, &s_lcnt, [&](int32_t p, uint32_t o) {
            if (o == kUnplacedT) {
                const uint32_t d = atomicAdd(&s_ndyn, 1u);
                if (d < T_DYN_CAP) {
                    dpos[d] = (uint32_t)p;
                    return;
                }
                // more late predecessors than other workgroups: the grid
                // broke its bound.  Report it; waiting here keeps the result
                // right and every workgroup finishing.
                raise_status(a.status, MP_EDEVICE);
                while ((o = agent_load(a.off + p)) == kUnplacedT) __builtin_amdgcn_s_sleep(2);
            }
            const uint32_t k = atomicAdd(&s_nstat, 1u);
            if (k < (uint32_t)stat_cap) gkeys[k] = ((uint64_t)o << 32) | (uint64_t)(o + a.su[p]);
        });
        __syncthreads();
        uint32_t nstat = s_nstat;
        const int ndyn = (int)min(s_ndyn, T_DYN_CAP);
        if (nstat > (uint32_t)stat_cap) {
            // more predecessors than the workgroup's buffer: wait for the late
            // ones, take a pool slot, collect every predecessor's range there
            // and fit over all of them (the general fit)
            for (int d = threadIdx.x; d < ndyn; d += BLOCK)
                while (agent_load(a.off + dpos[d]) == kUnplacedT) __builtin_amdgcn_s_sleep(1);
            __syncthreads();
            const uint32_t slot = pool_acquire(a.fl, &s_slot);
            const GenRanges gr = pool_ranges(a.pool, slot, a.n);
            if (threadIdx.x == 0) s_nstat = 0;
            __syncthreads();
            for_each_pred<BLOCK>(a, qt, st, lthr, n_long, band_list, &s_lcnt, [&](int32_t p, uint32_t o) {
                while (o == kUnplacedT) o = agent_load(a.off + p);  // placed: seen above
                const uint32_t k = atomicAdd(&s_nstat, 1u);
                gr.ks[k] = o;
                gr.ke[k] = (uint64_t)o + a.su[p];
            });
            __syncthreads();
            const uint64_t x = fit_general<BLOCK>(gr, s_nstat, st, T_BEST != 0, skeys,
                                                  skeys + kGRun, scratch64);
            pool_release(a.fl, slot);
            if (threadIdx.x == 0) agent_store(a.off + qt, (uint32_t)x);
            __syncthreads();
            continue;
        }
        // 2. sorted runs of the placed predecessors: one in LDS when it fits,
        //    else runs of kRunCap sorted in LDS and kept in global scratch
        // beyond a few hundred ranges the union is cheaper than a sort
        int nruns = (int)((nstat + kRunCap - 1) / kRunCap);
        uint32_t m_union = 0;
        if (nstat > kUnionMin && union_run<BLOCK>(gkeys, nstat, skeys, scratch, scratch64, &m_union)) {
            nstat = m_union;
            nruns = 1;
        } else if (nruns == 1) {
            for (int i = threadIdx.x; i < (int)nstat; i += BLOCK) skeys[i] = gkeys[i];
            __syncthreads();
            make_run<BLOCK>(skeys, (int)nstat, scratch);
        } else {
            for (int run = 0; run < nruns; ++run) {
                const int m0 = (int)min((uint32_t)kRunCap, nstat - (uint32_t)run * kRunCap);
                uint64_t* g = gkeys + (int64_t)run * kRunCap;
                for (int i = threadIdx.x; i < m0; i += BLOCK) skeys[i] = g[i];
                __syncthreads();
                make_run<BLOCK>(skeys, m0, scratch);
                for (int i = threadIdx.x; i < m0; i += BLOCK) g[i] = skeys[i];
                __syncthreads();
            }
        }
        // Lowest fit with one run of placed predecessors: before waiting,
        // mark the run's gaps [prefix maximum below i, start of i) that hold
        // t.  Then wave 0 alone waits for the late ones (all of them: one to
        // four a lane, their ranges stay in registers) and walks the
        // marked gaps in order, then the top: in a gap it moves past the
        // highest end among the late ranges overlapping [c, c + st) until
        // none does, and the first gap that still holds t gives the offset.
        // No workgroup barrier lies between the last wait and the publish.
        if (!T_BEST && nruns <= 1) {
            const int m = (int)nstat, words = (m + 63) >> 6;
            const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
            for (int w = wid; w < words; w += BLOCK / kWave) {
                const int i = 64 * w + lane;
                bool ok = false;
                if (i < m) {
                    const uint32_t g0 = i ? run_pmax(skeys[i - 1]) : 0u, g1 = run_start(skeys[i]);
                    ok = g1 > g0 && g1 - g0 >= st;
                }
                const uint64_t mk = __ballot(ok);
                if (lane == 0) gbits[w] = mk;
            }
            __syncthreads();
            // wave 0; K late predecessors a lane (K = 1, 4 or 8 for up to 64,
            // 256 or 512 of them)
            auto wave0 = [&](auto k_late) {
                constexpr int K = decltype(k_late)::value;
                // The first 64 marked gaps, in address order, one per lane
                // (a prefix count over the first 64 words of marks); a gap
                // beyond them is reached by the walk further down.
                const uint64_t my_bits = lane < words ? gbits[lane] : 0ull;
                const uint32_t my_cnt = (uint32_t)__popcll(my_bits);
                const uint32_t incl = wave_inclusive_sum(my_cnt);
                const uint32_t n_marked = (uint32_t)__shfl(incl, kWave - 1, kWave);
                const int ncand = (int)min(n_marked, (uint32_t)kWave);
                uint32_t slot = incl - my_cnt;
                for (uint64_t bm = my_bits; bm && slot < (uint32_t)kWave; bm &= bm - 1, ++slot)
                    cidx[slot] = (uint32_t)(64 * lane + __builtin_ctzll(bm));
                __builtin_amdgcn_wave_barrier();
                uint32_t cg0 = 0, cg1 = 0;  // this lane's candidate gap [cg0, cg1)
                if (lane < ncand) {
                    const int i = (int)cidx[lane];
                    cg0 = i ? run_pmax(skeys[i - 1]) : 0u;
                    cg1 = run_start(skeys[i]);
                }
                // marked gaps past the candidates: the walk resumes after the
                // last candidate (word 64 on when the first 64 words hold no more)
                const int resume = n_marked > (uint32_t)kWave || words > kWave
                                       ? (n_marked >= (uint32_t)kWave
                                              ? (int)(uint32_t)__builtin_amdgcn_readlane(
                                                    (int)cidx[kWave - 1], 0) + 1
                                              : 64 * kWave)
                                       : m;
                // When every marked gap is a candidate and a lane is left, that
                // lane holds the top of the run (no end): the walk then never
                // runs past the candidates.
                const bool closed = resume == m && ncand < kWave;
                const int nc = ncand + (closed ? 1 : 0), ktop = closed ? ncand : -1;
                if (closed && lane == ncand) cg0 = m ? run_pmax(skeys[m - 1]) : 0u;
                // this lane's late ranges (late predecessor lane + 64 r in
                // slot r), empty until known
                uint32_t lo_d[K], hi_d[K];
#pragma unroll
                for (int r = 0; r < K; ++r) {
                    lo_d[r] = kUnplacedT;
                    hi_d[r] = 0;
                }
                // lowest c' >= c with [c', c' + st) clear of every known late
                // range: jump to the highest end among the (few) overlapping ones
                auto past_late = [&](uint32_t c) {
                    while (true) {
                        uint32_t mx = 0;  // highest overlapping end of this lane (ends are > 0)
#pragma unroll
                        for (int r = 0; r < K; ++r)
                            mx = (lo_d[r] < c + st && c < hi_d[r]) ? max(mx, hi_d[r]) : mx;
                        uint64_t ov = __ballot(mx != 0);
                        if (!ov) return c;
                        uint32_t v = c;
                        for (; ov; ov &= ov - 1)
                            v = max(v, (uint32_t)__builtin_amdgcn_readlane((int)mx, (int)__builtin_ctzll(ov)));
                        c = v;
                    }
                };
                // lowest fit at or above c in candidates k on: x and its
                // candidate xk; false when it runs past the candidates
                uint32_t x = 0;
                int xk = 0;
                auto walk = [&](int k, uint32_t c) {
                    for (; k < nc; ++k) {
                        c = past_late(max(c, (uint32_t)__builtin_amdgcn_readlane((int)cg0, k)));
                        if (k == ktop ||
                            (uint64_t)c + st <= (uint32_t)__builtin_amdgcn_readlane((int)cg1, k)) {
                            x = c;
                            xk = k;
                            return true;
                        }
                    }
                    return false;
                };
                // The wait, one late predecessor a lane.  Known ranges only
                // raise the lowest fit, so the answer is kept up to date as
                // they arrive: it moves (the walk resumes from it) only when
                // a range that arrived overlaps it.
                uint32_t pend = 0, p[K], sp[K];  // pend: bit r for slot r
#pragma unroll
                for (int r = 0; r < K; ++r) {
                    const int d = lane + kWave * r;
                    p[r] = d < ndyn ? dpos[d] : 0u;
                    sp[r] = d < ndyn ? a.su[p[r]] : 0u;
                    pend |= d < ndyn ? 1u << r : 0u;
                }
                bool ok = walk(0, 0u);
                while (__ballot(pend != 0)) {
                    uint32_t o[K];
#pragma unroll
                    for (int r = 0; r < K; ++r) o[r] = (pend >> r) & 1u ? agent_load(a.off + p[r]) : kUnplacedT;
                    bool got = false, hit = false;
#pragma unroll
                    for (int r = 0; r < K; ++r) {
                        if (o[r] != kUnplacedT) {
                            lo_d[r] = o[r];
                            hi_d[r] = o[r] + sp[r];
                            pend &= ~(1u << r);
                            got = true;
                            hit = hit || (lo_d[r] < x + st && x < hi_d[r]);
                        }
                    }
                    // no sleep between polls: each takes an agent-scope load's
                    // round trip, and a sleep only delays the detection
                    if (!__ballot(got)) continue;
                    if (ok && __ballot(hit)) ok = walk(xk, x);
                }
                // every late range is known
                if (!ok) {  // past the candidates: the marked gaps after them, then the top
                    bool found = walk(0, 0u);
                    for (int w = resume >> 6; w < words && !found; ++w) {
                        uint64_t bm = gbits[w];
                        if (w == (resume >> 6)) bm &= ~0ull << (resume & 63);
                        for (; bm; bm &= bm - 1) {
                            const int i = 64 * w + __builtin_ctzll(bm);
                            const uint32_t g0 = i ? run_pmax(skeys[i - 1]) : 0u, g1 = run_start(skeys[i]);
                            const uint32_t c = past_late(g0);
                            if ((uint64_t)c + st <= g1) {
                                x = c;
                                found = true;
                                break;
                            }
                        }
                    }
                    if (!found) x = past_late(m ? run_pmax(skeys[m - 1]) : 0u);
                }
                if (lane == 0) agent_store(a.off + qt, x);
            };
            if (wid == 0) {
                if (T_WIDEST_WAIT) wave0(std::integral_constant<int, 8>{});
                else if (ndyn <= kWave) wave0(std::integral_constant<int, 1>{});
                else if (ndyn <= 4 * kWave) wave0(std::integral_constant<int, 4>{});
                else wave0(std::integral_constant<int, 8>{});
            }
            __syncthreads();
            continue;
        }
        // 3. wait for the predecessors that were not placed yet; their ranges
        //    form one more run
        for (int d = threadIdx.x; d < ndyn; d += BLOCK) {
            const uint32_t p = dpos[d];
            uint32_t o;
            while ((o = agent_load(a.off + p)) == kUnplacedT) __builtin_amdgcn_s_sleep(1);
            dkeys[d] = ((uint64_t)o << 32) | (uint64_t)(o + a.su[p]);
        }
        __syncthreads();
        if (ndyn) make_run<BLOCK>(dkeys, ndyn, scratch);
        // 4. the fit over every run (one pass)
        RunRef runs[kScratchRuns + 1];
        int nr = 0;
        if (nruns == 1) {
            runs[nr++] = RunRef{skeys, (int)nstat};
        } else {
            for (int run = 0; run < nruns; ++run)
                runs[nr++] = RunRef{gkeys + (int64_t)run * kRunCap,
                                    (int)min((uint32_t)kRunCap, nstat - (uint32_t)run * kRunCap)};
        }
        if (ndyn) runs[nr++] = RunRef{dkeys, ndyn};
        uint32_t x;
        if (T_BEST) x = best_fit_runs<BLOCK, kScratchRuns + 1>(runs, nr, st, scratch64);
        else x = nr ? fit_runs<BLOCK, kScratchRuns + 1>(runs, nr, st, scratch) : 0u;
        if (threadIdx.x == 0) agent_store(a.off + qt, x);
        __syncthreads();
    }
}

#undef T_DYN_CAP
#undef T_BEST
#undef T_WIDEST_WAIT

__global__ __launch_bounds__(256) void t_output_kernel(const uint32_t* __restrict__ off,
                                                       const uint32_t* __restrict__ su,
                                                       const uint64_t* __restrict__ off64,
                                                       const uint64_t* __restrict__ su64,
                                                       const uint32_t* __restrict__ pid, int64_t n,
                                                       int64_t* __restrict__ offset_out,
                                                       TFlags* fl, int64_t* __restrict__ peak_out) {
    __shared__ uint64_t red[256 / kWave];
    __shared__ uint32_t s_last;
    if (fl->abort) {
        if (blockIdx.x == 0 && threadIdx.x == 0) *peak_out = (int64_t)fl->peak;
        return;
    }
    const uint32_t sh = fl->shift;
    const bool wide = fl->wide != 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    uint64_t pk = 0;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n; q += stride) {
        const uint64_t o = wide ? off64[q] : (uint64_t)off[q];
        offset_out[pid[q]] = (int64_t)(o << sh);
        const uint64_t e = (o + (wide ? su64[q] : (uint64_t)su[q])) << sh;
        pk = pk > e ? pk : e;
    }
    pk = block_reduce<256>(pk, OpMax<uint64_t>(), red);
    if (threadIdx.x == 0) {
        if (pk) atomicMax(reinterpret_cast<unsigned long long*>(&fl->peak), (unsigned long long)pk);
        __threadfence();
        s_last = atomicAdd(&fl->done_output, 1u) == gridDim.x - 1 ? 1u : 0u;
    }
    __syncthreads();
    if (s_last && threadIdx.x == 0) {  // every workgroup's maximum is in
        __threadfence();
        *peak_out = (int64_t)flag_load64(&fl->peak);
    }
}

__global__ void t_peak_kernel(const TFlags* fl, int64_t* peak_out) { *peak_out = (int64_t)fl->peak; }


struct TLayout {
    size_t flags, su, pf, pl, pid, off, su64, off64, reach, keys0, vals0, keys1, vals1, radix,
        lflag, lpartial, llist, run_keys, pool, xbase, total;
    int64_t xcap;  // rank blocks an XCD can claim
    unsigned grid;
};

// Workgroups of the placement kernel on the current device: every resident
// one (more would only wait for a CU), at most 265 so that a tensor never
// has more late predecessors than wave 0 holds (the other workgroups' ranks
// and the untaken ranks of the other XCDs' current blocks).  The launch
// needs no co-residency -- a workgroup waits only on lower ranks, each held
// by a running workgroup or taken once one on its XCD finishes -- so this
// is a plain launch sized for throughput.
unsigned place_grid() {
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
        cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, t_place_kernel<kTBlock>, kTBlock, 0) !=
            hipSuccess ||
        per < 1)
        per = 1;
    const int64_t g = (int64_t)cus * per;
    constexpr int64_t kMaxGrid = kDynCap + 1 - kXcdGroups * ((int64_t)kTicketBlock - 1);
    static_assert(kMaxGrid >= 256, "one workgroup per CU of the largest device");
    return (unsigned)(g > kMaxGrid ? kMaxGrid : g);
}

// Keys per workgroup buffer: a tensor has fewer than n predecessors; the
// 64-bit path uses the same bytes as four arrays of stat_cap / 4 ranges.
int64_t stat_cap_of(int64_t n) {
    const int64_t cap = kScratchRuns * (int64_t)kRunCap;
    return 4 * n < cap ? 4 * n : cap;
}

TLayout t_layout(int64_t n, unsigned grid) {
    TLayout L{};
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += (bytes + 255) & ~(size_t)255;
        return at;
    };
    const int64_t nn = n > 0 ? n : 1;
    L.flags = take(sizeof(TFlags));
    L.su = take(nn * 4);
    L.pf = take(nn * 4);
    L.pl = take(nn * 4);
    L.pid = take(nn * 4);
    L.off = take(nn * 4);
    L.su64 = take(nn * 8);
    L.off64 = take(nn * 8);
    L.reach = take(nn * 4);
    L.keys0 = take(nn * 8);
    L.vals0 = take(nn * 4);
    L.keys1 = take(nn * 8);
    L.vals1 = take(nn * 4);
    L.radix = take(radix_workspace_bytes(nn));
    L.lflag = take(nn * 8);
    L.lpartial = take(scan_workspace_bytes(nn));
    L.llist = take(nn * 4);
    L.run_keys = take((size_t)grid * (size_t)stat_cap_of(nn) * 8);
    L.pool = take((size_t)kPoolSlots * 4 * nn * 8);
    // an XCD takes at most n ranks and one more per workgroup (the take
    // that ends it): blocks 0 .. (n + grid) / kTicketBlock
    L.xcap = (nn + (int64_t)grid) / kTicketBlock + 2;
    L.xbase = take((size_t)kXcdGroups * (size_t)L.xcap * 4);
    L.total = o;
    L.grid = grid;
    return L;
}

unsigned grid_n(int64_t n, int block) {
    const int64_t g = (n + block - 1) / block;
    return (unsigned)(g < 1 ? 1 : (g > 4096 ? 4096 : g));
}

}  // namespace

size_t plan_trace_workspace_bytes(int64_t n) { return t_layout(n, place_grid()).total; }

hipError_t launch_plan_trace(const int64_t* size, const int32_t* first, const int32_t* last,
                             int64_t n, int32_t num_ops, int32_t policy, int64_t* offset_out,
                             int64_t* peak_out, void* ws, int32_t* status, hipStream_t st) {
    const TLayout L = t_layout(n, place_grid());
    char* w = static_cast<char*>(ws);
    TFlags* fl = reinterpret_cast<TFlags*>(w + L.flags);
    uint32_t* su = reinterpret_cast<uint32_t*>(w + L.su);
    int32_t* pf = reinterpret_cast<int32_t*>(w + L.pf);
    int32_t* pl = reinterpret_cast<int32_t*>(w + L.pl);
    uint32_t* pid = reinterpret_cast<uint32_t*>(w + L.pid);
    uint32_t* off = reinterpret_cast<uint32_t*>(w + L.off);
    uint64_t* su64 = reinterpret_cast<uint64_t*>(w + L.su64);
    uint64_t* off64 = reinterpret_cast<uint64_t*>(w + L.off64);
    int32_t* reach = reinterpret_cast<int32_t*>(w + L.reach);
    uint64_t* keys0 = reinterpret_cast<uint64_t*>(w + L.keys0);
    uint32_t* vals0 = reinterpret_cast<uint32_t*>(w + L.vals0);
    uint64_t* keys1 = reinterpret_cast<uint64_t*>(w + L.keys1);
    uint32_t* vals1 = reinterpret_cast<uint32_t*>(w + L.vals1);
    void* rws = w + L.radix;
    int64_t* lflag = reinterpret_cast<int64_t*>(w + L.lflag);
    int64_t* lpartial = reinterpret_cast<int64_t*>(w + L.lpartial);
    int32_t* llist = reinterpret_cast<int32_t*>(w + L.llist);

    hipLaunchKernelGGL(t_init_kernel, dim3(1), dim3(64), 0, st, fl);
    if (n == 0) {
        hipLaunchKernelGGL(t_peak_kernel, dim3(1), dim3(1), 0, st, (const TFlags*)fl, peak_out);
        return hipGetLastError();
    }
    const unsigned g = grid_n(n, 256);
    uint32_t* xbase = reinterpret_cast<uint32_t*>(w + L.xbase);
    const int64_t nx = (int64_t)kXcdGroups * L.xcap;
    hipLaunchKernelGGL(t_ingest_kernel, dim3(g), dim3(256), 0, st, size, first, last, n, num_ops,
                       fl, status, keys0, vals0, xbase, nx);
    // position order (unsorted inputs only)
    bool alt = false;
    hipError_t e = radix_sort_pairs(keys0, vals0, keys1, vals1, n, 0, 32, rws, &alt, st,
                                    &fl->sorted);
    if (e != hipSuccess) return e;
    // positions, and the rank-sort pairs in (keys0, vals0)
    hipLaunchKernelGGL(t_positions_kernel, dim3(g), dim3(256), 0, st,
                       (const uint32_t*)(alt ? vals1 : vals0), size, first, last, n, su, pf, pl,
                       pid, off, su64, off64, keys0, vals0, (const TFlags*)fl);
    hipLaunchKernelGGL(t_reach_kernel, dim3(g), dim3(256), 0, st, first, last, (const int32_t*)pf,
                       (const int32_t*)pl, (const uint32_t*)pid, n, reach, fl);
    hipLaunchKernelGGL(t_long_flags_kernel, dim3(g), dim3(256), 0, st, (const int32_t*)reach, n,
                       lflag, (const TFlags*)fl);
    e = device_scan_i64(lflag, n, false, lpartial, nullptr, st, &fl->abort);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(t_long_list_kernel, dim3(g), dim3(256), 0, st, (const int32_t*)reach,
                       (const int64_t*)lflag, n, llist, fl);
    // rank order: size descending, stable over positions -- 32-bit keys, or
    // 64-bit ones when the unit counts are (the other sort is skipped on the
    // device; both take an even number of passes, so the result is in keys0)
    e = radix_sort_pairs(keys0, vals0, keys1, vals1, n, 0, 32, rws, &alt, st, &fl->skip_narrow);
    if (e != hipSuccess) return e;
    bool alt64 = false;
    e = radix_sort_pairs(keys0, vals0, keys1, vals1, n, 0, 64, rws, &alt64, st, &fl->skip_wide);
    if (e != hipSuccess) return e;
    if (alt != alt64) return hipErrorInvalidValue;  // both sorts end in the same buffer
    uint64_t* pool = reinterpret_cast<uint64_t*>(w + L.pool);
    PlaceArgs pa{su,
                 reach,
                 alt ? vals1 : vals0,
                 llist,
                 off,
                 reinterpret_cast<uint64_t*>(w + L.run_keys),
                 stat_cap_of(n),
                 pool,
                 n,
                 fl,
                 status,
                 policy == MP_BEST_FIT ? 1 : 0,
                 xbase,
                 L.xcap};
#ifdef MP_DEBUG_WAIT
    // test build: MEMOPLAN_DEBUG_WAIT=wide makes every wait hold eight late
    // predecessors a lane; =tight besides caps the late list at 8, so tensors
    // with more wait for the rest during the collection (and report
    // MP_EDEVICE, the condition that path exists for).  Offsets stay exact.
    if (const char* dbg = getenv("MEMOPLAN_DEBUG_WAIT")) {
        if (!strcmp(dbg, "wide")) pa.best |= 0x200;
        if (!strcmp(dbg, "tight")) pa.best |= 0x300;
    }
#endif
    hipLaunchKernelGGL(t_place_kernel<kTBlock>, dim3(L.grid), dim3(kTBlock), 0, st, pa);
    WideArgs wa{su64, reach, alt ? vals1 : vals0, llist, off64,
                reinterpret_cast<uint64_t*>(w + L.run_keys), stat_cap_of(n) / 4, pool, n, fl,
                policy == MP_BEST_FIT ? 1 : 0};
    hipLaunchKernelGGL(t_place_wide_kernel<kTBlock>, dim3(L.grid), dim3(kTBlock), 0, st, wa);
    hipLaunchKernelGGL(t_output_kernel, dim3(g), dim3(256), 0, st, (const uint32_t*)off,
                       (const uint32_t*)su, (const uint64_t*)off64, (const uint64_t*)su64,
                       (const uint32_t*)pid, n, offset_out, fl, peak_out);
    return hipGetLastError();
}

}  // namespace mp
