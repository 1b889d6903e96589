// Plan validation: every pair of tensors whose lifetimes intersect and whose
// byte ranges overlap (the pairwise ordering constraints of Eq. 2.1 state
// that such a pair may not exist in a valid plan).
//
// Works on one trace or on a batch of contiguous traces (segments).  Tensors
// are taken in position order (segment, first, id); for positions q < j of
// one segment the lifetimes meet iff first[j] <= last[q], so row q's
// candidates are the contiguous positions (q, reach[q]).  Short rows are
// handled by one thread each.  Long rows are sorted by band length (one
// class per power of two, stable, so ascending rows inside a class) and cut
// into chunks of 64; the count pass tests a chunk against tiles of 1024
// candidates staged in registers, so the long bands of a chunk share every
// load.  A device-wide scan of the row counts then gives each row its start,
// and the write pass visits only rows that have pairs, one workgroup per row
// in j order.  When the input is not already sorted by first inside each
// segment, positions come from a radix sort and the written pairs are
// radix-sorted at the end.
#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr int kVBlock = 256;
constexpr int32_t kShortRow = 64;  // longer rows go to the chunked kernels
constexpr unsigned kLongGrid = 1024;               // workgroups of the long rows' write pass
constexpr int kChunkRows = 64;                      // long rows per chunk (one per lane)
constexpr int kTileItems = 4;                       // candidates per thread per tile
constexpr int64_t kTileJ = kVBlock * kTileItems;    // candidates per tile
constexpr unsigned kTileGrid = 2048;                // workgroups of the count pass (tile ranges)
constexpr int kWriteUnroll = 8;                     // candidate loads in flight per lane (write pass)

// Workspace words.
struct VFlags {
    uint32_t unsorted;  // some segment is not sorted by first
    uint32_t sorted;    // == !unsorted (lets sort-path kernels skip themselves)
    uint32_t n_long;    // rows longer than kShortRow
    uint32_t wide;      // some offset + size is 2^32 or more
    int64_t begin1[2];  // {0, n} when the caller gives a single trace
};

struct VArrays {  // position-ordered views (inputs themselves when sorted)
    const int32_t* first;
    const int32_t* last;
    const int64_t* off;
    const int64_t* size;
    const uint32_t* id;  // null when sorted: id == position
};

__device__ __forceinline__ VArrays pick_arrays(const VFlags* fl, const int32_t* first,
                                               const int32_t* last, const int64_t* off,
                                               const int64_t* size, const int32_t* pf,
                                               const int32_t* pl, const int64_t* po,
                                               const int64_t* ps, const uint32_t* pid) {
    if (fl->unsorted) return VArrays{pf, pl, po, ps, pid};
    return VArrays{first, last, off, size, nullptr};
}

__global__ void v_init_kernel(VFlags* fl, int64_t n) {
    fl->unsorted = 0;
    fl->sorted = 1;
    fl->n_long = 0;
    fl->wide = 0;
    fl->begin1[0] = 0;
    fl->begin1[1] = n;
}

// Single trace: every tensor's segment ends at n.
__global__ void v_segend_one_kernel(int64_t n, int32_t* __restrict__ segend) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        segend[i] = (int32_t)n;
}

// Lanes below this one whose bit is set in m.
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Sort key of a row: floor(log2(band)) for long rows (band > kShortRow, so
// at least 6), 0 for short ones.
__device__ __forceinline__ uint64_t row_class(int64_t band) {
    return band > kShortRow ? (uint64_t)(63 - __clzll(band)) : 0;
}

// Segment end of every tensor, and checks of the segment table.
__global__ void v_segend_kernel(const int64_t* __restrict__ begin, int64_t n_seg, int64_t n,
                                int32_t* __restrict__ segend, int32_t* __restrict__ status) {
    for (int64_t b = blockIdx.x; b < n_seg; b += gridDim.x) {
        const int64_t lo = begin[b], hi = begin[b + 1];
        if (lo < 0 || hi < lo || hi > n || (b == 0 && lo != 0) || (b == n_seg - 1 && hi != n)) {
            if (threadIdx.x == 0) raise_status(status, MP_EINVAL);
            continue;
        }
        for (int64_t i = lo + threadIdx.x; i < hi; i += blockDim.x) segend[i] = (int32_t)hi;
    }
}

__global__ __launch_bounds__(kVBlock) void v_check_kernel(
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, const int64_t* __restrict__ off, int64_t n,
    const int32_t* __restrict__ segend, VFlags* fl, int32_t* __restrict__ status,
    int assume_sorted) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    bool bad = false, unsorted = false, wide = false;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int64_t s = size[i], o = off[i];
        const int32_t f = first[i], l = last[i];
        if (s <= 0 || f < 0 || f > l || o < 0 || o > INT64_MAX - s) bad = true;
        else if (o + s > (int64_t)UINT32_MAX) wide = true;
        if (i + 1 < n && i + 1 < segend[i] && first[i + 1] < f) unsorted = true;
    }
    if (__ballot(bad) && (threadIdx.x & (kWave - 1)) == 0) raise_status(status, MP_EINVAL);
    if (__ballot(wide) && (threadIdx.x & (kWave - 1)) == 0) atomicOr(&fl->wide, 1u);
    if (__ballot(unsorted) && (threadIdx.x & (kWave - 1)) == 0) {
        if (assume_sorted) {  // broken promise: report, stay on the sorted path
            raise_status(status, MP_EINVAL);
        } else {
            atomicOr(&fl->unsorted, 1u);
            atomicAnd(&fl->sorted, 0u);
        }
    }
}

// Unsorted inputs only: sort keys (segment end, first) with the index.
__global__ void v_keys_kernel(const int32_t* __restrict__ first, const int32_t* __restrict__ segend,
                              int64_t n, uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
                              const VFlags* fl) {
    if (!fl->unsorted) return;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        keys[i] = ((uint64_t)(uint32_t)segend[i] << 32) | (uint32_t)first[i];
        vals[i] = (uint32_t)i;
    }
}

__global__ void v_gather_kernel(const uint32_t* __restrict__ perm, const int64_t* __restrict__ size,
                                const int32_t* __restrict__ first, const int32_t* __restrict__ last,
                                const int64_t* __restrict__ off, int64_t n, int32_t* __restrict__ pf,
                                int32_t* __restrict__ pl, int64_t* __restrict__ po,
                                int64_t* __restrict__ ps, uint32_t* __restrict__ pid,
                                const VFlags* fl) {
    if (!fl->unsorted) return;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n; q += stride) {
        const uint32_t i = perm[q];
        pf[q] = first[i];
        pl[q] = last[i];
        po[q] = off[i];
        ps[q] = size[i];
        pid[q] = i;
    }
}

// reach[q]: first position of q's segment after q whose first op is > last[q].
__device__ __forceinline__ int32_t find_reach(const int32_t* f, int32_t q, int32_t end, int32_t l) {
    int32_t known = q, step = 1, probe = q + 1;
    while (probe < end && f[probe] <= l) {
        known = probe;
        step <<= 1;
        probe = q + step;
    }
    int32_t a = known + 1, z = probe < end ? probe : end;
    while (a < z) {
        const int32_t mid = a + ((z - a) >> 1);
        if (f[mid] <= l) a = mid + 1;
        else z = mid;
    }
    return a;
}

__device__ __forceinline__ bool bytes_meet(int64_t oa, int64_t sa, int64_t ob, int64_t sb) {
    return oa < ob + sb && ob < oa + sa;
}

__device__ __forceinline__ void put_pair(int64_t* pairs, int64_t pos, int64_t cap, const VArrays& a,
                                         int64_t q, int64_t j) {
    if (pos >= cap) return;
    int64_t x = a.id ? (int64_t)a.id[q] : q, y = a.id ? (int64_t)a.id[j] : j;
    if (x > y) {
        const int64_t t = x;
        x = y;
        y = t;
    }
    pairs[2 * pos] = x;
    pairs[2 * pos + 1] = y;
}

// Pass over short rows (one thread per row).
//   write == 0: cnt[q] = conflicts of row q (0 for long rows), reach[q]
//               stored, (class, q) written as a sort key and value, long rows
//               counted
//   write == 1: pairs of row q written from cnt[q] (now its start)
__global__ __launch_bounds__(kVBlock) void v_rows_kernel(
    const int32_t* first, const int32_t* last, const int64_t* off, const int64_t* size,
    const int32_t* pf, const int32_t* pl, const int64_t* po, const int64_t* ps,
    const uint32_t* pid, const int32_t* __restrict__ segend, int64_t n, int32_t* __restrict__ reach,
    int64_t* __restrict__ cnt, uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
    VFlags* fl, int write, int64_t* __restrict__ pairs, int64_t cap) {
    const VArrays a = pick_arrays(fl, first, last, off, size, pf, pl, po, ps, pid);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n; q += stride) {
        int32_t r;
        if (!write) {
            // clamp the segment end so that a rejected segment table stays in bounds
            int64_t end = segend[q];
            end = end > n ? n : (end < q + 1 ? q + 1 : end);
            r = find_reach(a.first, (int32_t)q, (int32_t)end, a.last[q]);
            reach[q] = r;
        } else {
            r = reach[q];
        }
        const int64_t band = (int64_t)r - q - 1;
        const bool is_long = band > kShortRow;
        if (!write) {
            keys[q] = row_class(band);
            vals[q] = (uint32_t)q;
            const uint64_t m = __ballot(is_long);
            if (m && (int)(threadIdx.x & (kWave - 1)) == __ffsll((unsigned long long)__ballot(1)) - 1)
                atomicAdd(&fl->n_long, (uint32_t)__popcll(m));
        }
        if (is_long) {
            if (!write) cnt[q] = 0;
            continue;
        }
        if (write && (cnt[q + 1] == cnt[q] || cnt[q] >= cap)) continue;  // nothing to write
        const int64_t oq = a.off[q], sq = a.size[q];
        int64_t pos = write ? cnt[q] : 0;
        for (int64_t j = q + 1; j < r; ++j) {
            if (bytes_meet(oq, sq, a.off[j], a.size[j])) {
                if (write) put_pair(pairs, pos, cap, a, q, j);
                ++pos;
            }
        }
        if (!write) cnt[q] = pos;
    }
}

// The long rows in class order are the last n_long values of the class sort.
__device__ __forceinline__ const uint32_t* long_rows_of(const uint32_t* sorted, int64_t n,
                                                        const VFlags* fl) {
    return sorted + (n - (int64_t)fl->n_long);
}

// Candidate range of every chunk of kChunkRows long rows (one wave per
// chunk): lo = smallest row + 1, tiles = ceil((largest reach - lo) / kTileJ).
__global__ __launch_bounds__(kVBlock) void v_chunk_kernel(const uint32_t* __restrict__ sorted,
                                                          int64_t n,
                                                          const int32_t* __restrict__ reach,
                                                          const VFlags* fl, int64_t n_chunk_max,
                                                          int32_t* __restrict__ chunk_lo,
                                                          int64_t* __restrict__ chunk_tiles) {
    const int64_t c = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
    if (c >= n_chunk_max) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t n_long = fl->n_long;
    const uint32_t* long_rows = long_rows_of(sorted, n, fl);
    const int64_t k = c * kChunkRows + lane;
    int32_t q = INT32_MAX, r = 0;
    if (k < n_long) {
        q = (int32_t)long_rows[k];
        r = reach[q];
    }
    const int32_t qmin = wave_reduce(q, OpMin<int32_t>());
    const int32_t rmax = wave_reduce(r, OpMax<int32_t>());
    if (lane == 0) {
        const bool any = c * kChunkRows < n_long;
        chunk_lo[c] = any ? qmin + 1 : 0;
        chunk_tiles[c] = any ? ((int64_t)rmax - (qmin + 1) + kTileJ - 1) / kTileJ : 0;
    }
}

__device__ __forceinline__ int64_t readlane64(int64_t v, int k) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, k);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), k);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ uint32_t readlane64(uint32_t v, int k) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, k);
}

// Byte ranges as T: int64_t, or uint32_t when every end is below 2^32.
template <typename T>
struct TileRows {
    int32_t q = INT32_MAX, r = 0;  // this lane's row of the chunk and its reach
    T o = 0, e = 0;                // and its byte range [o, e)
};

// One tile for one wave: kTileItems candidates per lane at j0 + i * 256 + tid
// against the rows of the chunk whose bands meet the tile (a ballot over the
// lanes that hold the rows; sentinel lanes have r = 0).  Row values are
// broadcast with readlane.  A row of a valid plan has no hits, so the test
// only ORs the hit masks; a row with hits is counted again exactly and one
// lane adds the count to cnt[q].
template <typename T>
__device__ __forceinline__ void tile_rows(const TileRows<T>& R, int64_t j0, int64_t n,
                                          const VArrays& a, int64_t* __restrict__ cnt) {
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    T jo[kTileItems], je[kTileItems];
    int32_t jj[kTileItems];
#pragma unroll
    for (int i = 0; i < kTileItems; ++i) {
        const int64_t j = j0 + i * kVBlock + tid;
        jj[i] = j < n ? (int32_t)j : INT32_MAX;  // past n: outside every band
        jo[i] = 0;
        je[i] = 0;
        if (j < n) {
            const int64_t o = a.off[j];
            jo[i] = (T)o;
            je[i] = (T)(o + a.size[j]);
        }
    }
    // tile [jlo, jhi) in int32 (jhi clamped; positions are below 2^31 - 1)
    const int32_t jlo = (int32_t)j0;
    const int32_t jhi = (int32_t)(j0 + kTileJ < INT32_MAX ? j0 + kTileJ : INT32_MAX);
    uint64_t act = __builtin_amdgcn_ballot_w64(R.r > jlo && R.q < jhi - 1);
    const uint64_t cover = __builtin_amdgcn_ballot_w64(R.q < jlo && R.r >= jhi);
    while (act) {
        const int k = (int)__builtin_ctzll(act);
        act &= act - 1;
        const T o = readlane64(R.o, k), e = readlane64(R.e, k);
        uint64_t any = 0;
        if ((cover >> k) & 1) {  // the band covers the tile (all of it below n)
#pragma unroll
            for (int i = 0; i < kTileItems; ++i)
                any |= __builtin_amdgcn_ballot_w64(o < je[i]) &
                       __builtin_amdgcn_ballot_w64(jo[i] < e);
        } else {
            const int32_t q = __builtin_amdgcn_readlane(R.q, k);
            const int32_t r = __builtin_amdgcn_readlane(R.r, k);
#pragma unroll
            for (int i = 0; i < kTileItems; ++i)
                any |= __builtin_amdgcn_ballot_w64(jj[i] > q) &
                       __builtin_amdgcn_ballot_w64(jj[i] < r) &
                       __builtin_amdgcn_ballot_w64(o < je[i]) &
                       __builtin_amdgcn_ballot_w64(jo[i] < e);
        }
        if (any) {
            const int32_t q = __builtin_amdgcn_readlane(R.q, k);
            const int32_t r = __builtin_amdgcn_readlane(R.r, k);
            uint32_t hits = 0;
#pragma unroll
            for (int i = 0; i < kTileItems; ++i)
                hits += (uint32_t)__popcll(__builtin_amdgcn_ballot_w64(
                    jj[i] > q && jj[i] < r && o < je[i] && jo[i] < e));
            if (lane == 0)
                atomicAdd(reinterpret_cast<unsigned long long*>(&cnt[q]),
                          (unsigned long long)hits);
        }
    }
}

// Count pass of the long rows.  tile_end is the inclusive prefix of the
// chunks' tile counts; the tiles are dealt to the workgroups in contiguous
// ranges.  Every wave works alone: it holds the chunk's rows one per lane
// and kTileItems candidates per lane of each tile.
template <typename T>
__device__ __forceinline__ void tile_pass(const VArrays& a, const int32_t* __restrict__ reach,
                                          const uint32_t* long_rows, int64_t n_long,
                                          const int32_t* __restrict__ chunk_lo,
                                          const int64_t* __restrict__ tile_end, int64_t n,
                                          int64_t c, int64_t t0, int64_t t1,
                                          int64_t* __restrict__ cnt) {
    const int lane = threadIdx.x & (kWave - 1);
    TileRows<T> R;
    int64_t loaded = -1;
    for (int64_t t = t0; t < t1; ++t) {
        while (tile_end[c] <= t) ++c;
        if (c != loaded) {
            R = TileRows<T>{};
            const int64_t k = c * kChunkRows + lane;
            if (k < n_long) {
                R.q = (int32_t)long_rows[k];
                R.r = reach[R.q];
                const int64_t o = a.off[R.q];
                R.o = (T)o;
                R.e = (T)(o + a.size[R.q]);
            }
            loaded = c;
        }
        tile_rows<T>(R, chunk_lo[c] + (t - (c ? tile_end[c - 1] : 0)) * kTileJ, n, a, cnt);
    }
}

__global__ __launch_bounds__(kVBlock) void v_tile_kernel(
    const int32_t* first, const int32_t* last, const int64_t* off, const int64_t* size,
    const int32_t* pf, const int32_t* pl, const int64_t* po, const int64_t* ps,
    const uint32_t* pid, const int32_t* __restrict__ reach, const uint32_t* __restrict__ sorted,
    const int32_t* __restrict__ chunk_lo, const int64_t* __restrict__ tile_end, int64_t n,
    const VFlags* fl, int64_t* __restrict__ cnt) {
    __shared__ int64_t s_chunk;
    const VArrays a = pick_arrays(fl, first, last, off, size, pf, pl, po, ps, pid);
    const int64_t n_long = fl->n_long;
    const uint32_t* long_rows = long_rows_of(sorted, n, fl);
    const int64_t n_chunks = (n_long + kChunkRows - 1) / kChunkRows;
    if (n_chunks == 0) return;
    const int64_t total = tile_end[n_chunks - 1];
    const int64_t t0 = total * blockIdx.x / gridDim.x, t1 = total * (blockIdx.x + 1) / gridDim.x;
    if (t0 >= t1) return;
    const int lane = threadIdx.x & (kWave - 1);
    if (threadIdx.x < kWave) {
        // first chunk whose tiles end after t0: 64-way search (tile_end[n_chunks-1] > t0)
        int64_t lo = 0, hi = n_chunks;
        while (hi - lo > 1) {
            const int64_t step = (hi - lo + kWave - 1) / kWave;
            const int64_t idx = lo + (lane + 1) * step - 1;
            const bool past = idx >= hi - 1 || tile_end[idx] > t0;
            const int f = __ffsll((unsigned long long)__ballot(past)) - 1;
            const int64_t nlo = lo + f * step;
            hi = nlo + step < hi ? nlo + step : hi;
            lo = nlo;
        }
        if (lane == 0) s_chunk = lo;
    }
    __syncthreads();
    if (fl->wide)
        tile_pass<int64_t>(a, reach, long_rows, n_long, chunk_lo, tile_end, n, s_chunk, t0, t1, cnt);
    else
        tile_pass<uint32_t>(a, reach, long_rows, n_long, chunk_lo, tile_end, n, s_chunk, t0, t1,
                            cnt);
}

// Write pass of the long rows that have pairs.  The workgroup checks 256 of
// its long rows at once (rows b, b + G, b + 2G, ... for workgroup b of G, so
// that neighbours in class order, often alike, land in different
// workgroups) and lists those with pairs; then each listed row is
// written by the whole workgroup: each wave takes a contiguous quarter of the
// band, counts its hits, and after an exchange of the four counts writes them
// in j order.  Rows write disjoint ranges, so the list order is free.
__global__ __launch_bounds__(kVBlock) void v_long_write_kernel(
    const int32_t* first, const int32_t* last, const int64_t* off, const int64_t* size,
    const int32_t* pf, const int32_t* pl, const int64_t* po, const int64_t* ps,
    const uint32_t* pid, const int32_t* __restrict__ reach, const int64_t* __restrict__ cnt,
    const uint32_t* __restrict__ sorted, int64_t n, const VFlags* fl,
    int64_t* __restrict__ pairs, int64_t cap) {
    constexpr int kWaves = kVBlock / kWave;
    __shared__ uint32_t wcnt[2][kWaves];
    __shared__ int32_t list[kVBlock];
    __shared__ uint32_t n_list;
    const VArrays a = pick_arrays(fl, first, last, off, size, pf, pl, po, ps, pid);
    const int64_t n_long = fl->n_long;
    const uint32_t* long_rows = long_rows_of(sorted, n, fl);
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    int buf = 0;
    const int64_t G = gridDim.x;
    for (int64_t base = blockIdx.x; base < n_long; base += G * kVBlock) {
        if (tid == 0) n_list = 0;
        __syncthreads();
        const int64_t k = base + tid * G;
        if (k < n_long) {
            const int32_t q = (int32_t)long_rows[k];
            const int64_t start = cnt[q];
            if (start != cnt[q + 1] && start < cap) list[atomicAdd(&n_list, 1u)] = q;
        }
        __syncthreads();
        const uint32_t listed = n_list;
        for (uint32_t li = 0; li < listed; ++li) {
            const int64_t q = list[li];
            const int64_t start = cnt[q];
            const int64_t r = reach[q];
            const int64_t oq = a.off[q], sq = a.size[q];
            const int64_t seg = ((r - q - 1 + kWaves * kWave - 1) / (kWaves * kWave)) * kWave;
            const int64_t s0 = q + 1 + wid * seg;
            const int64_t s1 = s0 + seg < r ? s0 + seg : r;
            uint32_t mine = 0;
            for (int64_t j0 = s0; j0 < s1; j0 += kWave * kWriteUnroll) {
                int64_t jo[kWriteUnroll], js[kWriteUnroll];  // all loads first, then the tests
#pragma unroll
                for (int u = 0; u < kWriteUnroll; ++u) {
                    const int64_t j = j0 + u * kWave + lane;
                    jo[u] = j < s1 ? a.off[j] : 0;
                    js[u] = j < s1 ? a.size[j] : 0;
                }
#pragma unroll
                for (int u = 0; u < kWriteUnroll; ++u) {
                    const int64_t j = j0 + u * kWave + lane;
                    mine += (uint32_t)__popcll(__ballot(j < s1 && bytes_meet(oq, sq, jo[u], js[u])));
                }
            }
            if (lane == 0) wcnt[buf][wid] = mine;
            __syncthreads();
            int64_t pos = start;
            for (int w = 0; w < wid; ++w) pos += wcnt[buf][w];
            buf ^= 1;  // the next row's exchange uses the other buffer
            for (int64_t j0 = s0; mine > 0 && j0 < s1; j0 += kWave * kWriteUnroll) {
                int64_t jo[kWriteUnroll], js[kWriteUnroll];
#pragma unroll
                for (int u = 0; u < kWriteUnroll; ++u) {
                    const int64_t j = j0 + u * kWave + lane;
                    jo[u] = j < s1 ? a.off[j] : 0;
                    js[u] = j < s1 ? a.size[j] : 0;
                }
#pragma unroll
                for (int u = 0; u < kWriteUnroll; ++u) {
                    const int64_t j = j0 + u * kWave + lane;
                    const bool h = j < s1 && bytes_meet(oq, sq, jo[u], js[u]);
                    const uint64_t m = __ballot(h);
                    if (h) put_pair(pairs, pos + lanes_below(m), cap, a, q, j);
                    pos += __popcll(m);
                    mine -= (uint32_t)__popcll(m);
                }
            }
        }
        __syncthreads();  // the list and n_list are rewritten for the next rows
    }
}

// ---- unsorted inputs with more pairs than the capacity
// The write pass keeps the first `cap` pairs of position order, which for an
// input not sorted by first are not the lexicographically first ones.  One
// workgroup then selects those: pair keys (smaller id << nbits | larger id)
// are unique, so the cap-th smallest key K* is found digit by digit from the
// top (12 bits at a time, histograms in LDS over the pairs whose key carries
// the digits chosen so far), and pairs[0, cap) is rewritten with the keys at
// or below K*; the pair sort that follows orders them.  Only rows with pairs
// are walked (row q has cnt[q + 1] - cnt[q], and its walk stops at the last).

constexpr int kSelBlock = 1024;
constexpr int kSelDigit = 12;
constexpr int kSelBins = 1 << kSelDigit;
constexpr int kSelUnroll = 4;

// f(key, x, y) for every pair (x < y ids) of every row with pairs; the
// workgroup's waves take 64 rows at a time.
template <class F>
__device__ __forceinline__ void sel_for_each_pair(const VArrays& a, const int32_t* reach,
                                                  const int64_t* cnt, int64_t n, int nbits, F f) {
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    constexpr int kWaves = kSelBlock / kWave;
    for (int64_t r0 = (int64_t)wid * kWave; r0 < n; r0 += (int64_t)kWaves * kWave) {
        const int64_t rq = r0 + lane;
        uint64_t rows = __ballot(rq < n && cnt[rq + 1] > cnt[rq]);
        while (rows) {
            const int64_t q = r0 + (__ffsll((unsigned long long)rows) - 1);
            rows &= rows - 1;
            const int64_t need = cnt[q + 1] - cnt[q];
            const int64_t r = reach[q];
            const int64_t oq = a.off[q], sq = a.size[q];
            const uint64_t xq = a.id ? (uint64_t)a.id[q] : (uint64_t)q;
            int64_t found = 0;
            for (int64_t j0 = q + 1; j0 < r && found < need; j0 += kWave * kSelUnroll) {
                int64_t jo[kSelUnroll], js[kSelUnroll];
#pragma unroll
                for (int u = 0; u < kSelUnroll; ++u) {
                    const int64_t j = j0 + u * kWave + lane;
                    jo[u] = j < r ? a.off[j] : 0;
                    js[u] = j < r ? a.size[j] : 0;
                }
#pragma unroll
                for (int u = 0; u < kSelUnroll; ++u) {
                    const int64_t j = j0 + u * kWave + lane;
                    const bool h = j < r && bytes_meet(oq, sq, jo[u], js[u]);
                    if (h) {
                        uint64_t x = xq, y = a.id ? (uint64_t)a.id[j] : (uint64_t)j;
                        if (x > y) {
                            const uint64_t t = x;
                            x = y;
                            y = t;
                        }
                        f((x << nbits) | y, x, y);
                    }
                    found += __popcll(__ballot(h));
                }
            }
        }
    }
}

__global__ __launch_bounds__(kSelBlock) void v_select_kernel(
    const int32_t* first, const int32_t* last, const int64_t* off, const int64_t* size,
    const int32_t* pf, const int32_t* pl, const int64_t* po, const int64_t* ps,
    const uint32_t* pid, const int32_t* __restrict__ reach, const int64_t* __restrict__ cnt,
    int64_t n, const VFlags* fl, const int64_t* __restrict__ n_out, int64_t cap, int nbits,
    int64_t* __restrict__ pairs) {
    __shared__ unsigned long long hist[kSelBins];
    __shared__ unsigned long long part[kSelBlock];
    __shared__ uint64_t s_prefix;
    __shared__ int64_t s_rank;
    __shared__ unsigned long long s_slot;
    if (!fl->unsorted || cap <= 0 || *n_out <= cap) return;
    const VArrays a = pick_arrays(fl, first, last, off, size, pf, pl, po, ps, pid);
    const int tid = threadIdx.x;
    constexpr int kPer = kSelBins / kSelBlock;
    uint64_t prefix = 0;  // the digits of K* chosen so far
    int64_t rank = cap;   // K* is the rank-th smallest key with that prefix (from 1)
    for (int top = 2 * nbits; top > 0;) {
        const int D = top < kSelDigit ? top : kSelDigit;
        const int shift = top - D;
        const uint64_t dmask = ((uint64_t)1 << D) - 1;
        for (int i = tid; i < kSelBins; i += kSelBlock) hist[i] = 0;
        __syncthreads();
        sel_for_each_pair(a, reach, cnt, n, nbits, [&](uint64_t key, uint64_t, uint64_t) {
            if ((key >> top) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1ull);
        });
        __syncthreads();
        // exclusive sums of the per-thread bin groups (Hillis-Steele), then the
        // thread whose bins hold the rank-th key names the digit
        unsigned long long mine = 0;
#pragma unroll
        for (int k = 0; k < kPer; ++k) mine += hist[tid * kPer + k];
        part[tid] = mine;
        __syncthreads();
        for (int d = 1; d < kSelBlock; d <<= 1) {
            const unsigned long long add = tid >= d ? part[tid - d] : 0ull;
            __syncthreads();
            part[tid] += add;
            __syncthreads();
        }
        int64_t before = (int64_t)(part[tid] - mine);
        if (before < rank && rank <= before + (int64_t)mine) {
            for (int k = 0; k < kPer; ++k) {
                const int64_t c = (int64_t)hist[tid * kPer + k];
                if (rank <= before + c) {
                    s_prefix = (prefix << D) | (uint64_t)(tid * kPer + k);
                    s_rank = rank - before;
                    break;
                }
                before += c;
            }
        }
        __syncthreads();
        prefix = s_prefix;
        rank = s_rank;
        top = shift;
        __syncthreads();  // s_prefix and s_rank are written again next digit
    }
    if (tid == 0) s_slot = 0;
    __syncthreads();
    const uint64_t kstar = prefix;
    sel_for_each_pair(a, reach, cnt, n, nbits, [&](uint64_t key, uint64_t x, uint64_t y) {
        if (key <= kstar) {
            const unsigned long long at = atomicAdd(&s_slot, 1ull);
            if ((int64_t)at < cap) {
                pairs[2 * at] = (int64_t)x;
                pairs[2 * at + 1] = (int64_t)y;
            }
        }
    });
}

__global__ void v_total_kernel(const int64_t* __restrict__ partial, int64_t tiles, int64_t cap,
                               int64_t* __restrict__ n_out, int32_t* __restrict__ status,
                               int64_t* __restrict__ cnt_end) {
    const int64_t total = partial[tiles];
    *n_out = total;
    if (cnt_end) *cnt_end = total;  // row starts then bound every row: cnt[q + 1] - cnt[q]
    if (total > cap) raise_status(status, MP_ENOSPC);
}

// Unsorted inputs: pack the written pairs into sort keys (i << nbits | j,
// ids below 2^nbits; unused slots all ones, so they sort last).
__global__ void v_pack_kernel(const int64_t* __restrict__ pairs, const int64_t* __restrict__ n_out,
                              int64_t cap, int nbits, uint64_t* __restrict__ keys,
                              const VFlags* fl) {
    if (!fl->unsorted) return;
    const int64_t m = *n_out < cap ? *n_out : cap;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < cap; k += stride)
        keys[k] = k < m ? (((uint64_t)pairs[2 * k] << nbits) | (uint64_t)pairs[2 * k + 1]) : ~0ull;
}

__global__ void v_unpack_kernel(const uint64_t* __restrict__ keys, const int64_t* __restrict__ n_out,
                                int64_t cap, int nbits, int64_t* __restrict__ pairs,
                                const VFlags* fl) {
    if (!fl->unsorted) return;
    const int64_t m = *n_out < cap ? *n_out : cap;
    const uint64_t low = ((uint64_t)1 << nbits) - 1;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < m; k += stride) {
        pairs[2 * k] = (int64_t)(keys[k] >> nbits);
        pairs[2 * k + 1] = (int64_t)(keys[k] & low);
    }
}

// ---- batches of short sorted traces: one workgroup per trace, the trace in LDS.
// Positions are ids (the caller promises first non-decreasing inside every
// trace); row q's candidates are (q, reach[q]).  The pairs of a trace are
// split evenly over the threads by pair index (row-major), so the count pass
// and the write pass enumerate the same pairs in (i, j) order.

constexpr int kVbBlock = 512;
constexpr int64_t kVbFuseMax = 4096;  // traces up to which the write pass sums the counts itself

// write == 0: segcnt[b] = conflicts of trace b.
// write == 1: segcnt holds exclusive starts (segcnt[n_seg] = total); the
//             pairs of trace b are written from segcnt[b] on, below `cap`.
template <int BLOCK, int ITEMS>
__global__ __launch_bounds__(BLOCK, ITEMS <= 4 ? 8 : 4) void vb_kernel(
    const int64_t* __restrict__ begin, int64_t n_seg, const int64_t* __restrict__ size,
    const int32_t* __restrict__ first, const int32_t* __restrict__ last,
    const int64_t* __restrict__ off, int64_t n, int32_t cap_n, int64_t* __restrict__ segcnt,
    int write, int64_t* __restrict__ pairs, int64_t cap, int64_t* __restrict__ n_out,
    int32_t* __restrict__ status) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ uint32_t scratch[BLOCK / kWave];
    __shared__ uint64_t scratch64[BLOCK / kWave];
    // LDS: first[N] i32 (reach search) -> then off[N], size[N] i64 over it;
    // band lengths -> starts [N+1] u32 after them.  20 bytes per tensor, so
    // four workgroups of 2000-tensor traces share a CU.
    const size_t N = (size_t)cap_n;
    int32_t* lf = reinterpret_cast<int32_t*>(smem);
    int64_t* lo64 = reinterpret_cast<int64_t*>(smem);
    int64_t* ls64 = reinterpret_cast<int64_t*>(smem + 8 * N);
    uint32_t* band = reinterpret_cast<uint32_t*>(smem + 16 * N);
    const int tid = threadIdx.x;
    for (int64_t b = blockIdx.x; b < n_seg; b += gridDim.x) {
        // write 2 (short batches): the counts are as the count pass left
        // them; this trace's first pair goes after the sum of those before
        // it, and the last trace's workgroup reports the total
        int64_t before = 0;
        if (write == 2) {
            uint64_t part = 0;
            for (int64_t i = tid; i < b; i += BLOCK) part += (uint64_t)segcnt[i];
            before = (int64_t)block_reduce<BLOCK>(part, OpAdd<uint64_t>(), scratch64);
            if (b == n_seg - 1 && tid == 0) {
                const int64_t total = before + segcnt[b];
                *n_out = total;
                if (total > cap) raise_status(status, MP_ENOSPC);
            }
        }
        const int64_t lo = begin[b], hi = begin[b + 1];
        if (lo < 0 || hi < lo || hi > n || (b == 0 && lo != 0) || (b == n_seg - 1 && hi != n) ||
            hi - lo > cap_n) {
            if (tid == 0) {
                raise_status(status, MP_EINVAL);
                if (!write) segcnt[b] = 0;
            }
            continue;
        }
        int64_t base = 0;
        if (write == 1) {
            base = segcnt[b];
            if (segcnt[b + 1] == base || base >= cap) continue;  // nothing to write here
        } else if (write == 2) {
            base = before;
            if (segcnt[b] == 0 || base >= cap) continue;
        }
        const int m = (int)(hi - lo);
        // first and last of every item are requested before any is used
        // (indices clamped into the trace: no branch around the loads)
        int32_t l_r[ITEMS];
        bool bad = false;
        {
            int32_t f_r[ITEMS];
            const int mc = m > 0 ? m - 1 : 0;
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                const int q = min(tid + k * BLOCK, mc);
                f_r[k] = m > 0 ? first[lo + q] : 0;
                l_r[k] = m > 0 ? last[lo + q] : 0;
            }
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                const int q = tid + k * BLOCK;
                if (q < m) {
                    if (f_r[k] < 0 || f_r[k] > l_r[k]) bad = true;
                    lf[q] = f_r[k];
                }
            }
        }
        __syncthreads();
        // reach.  When the trace's first ops span at most 3 N values, from a
        // table over them in the LDS the byte ranges take later: tab[v - f0]
        // = positions whose first op is at most v, so reach[q] =
        // tab[last[q] - f0] (every position when last[q] >= the highest
        // first op), clamped into (q, m] should the sorted promise be broken
        // (it is reported below).  Otherwise the next four positions are
        // probed at once (short bands end there) and longer bands gallop on.
        const int32_t f_lo = m > 0 ? lf[0] : 0, f_hi = m > 0 ? lf[m - 1] : 0;
        const bool use_tab = m > 0 && f_hi >= f_lo && (int64_t)f_hi - f_lo < 3 * (int64_t)N;
        uint32_t* tab = reinterpret_cast<uint32_t*>(smem + 4 * N);
        if (use_tab) {
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                const int q = tid + k * BLOCK;
                if (q < m) {
                    const int64_t f = lf[q], f1 = q + 1 < m ? lf[q + 1] : (int64_t)f_hi + 1;
                    for (int64_t v = f > f_lo ? f : f_lo; v < f1 && v <= f_hi; ++v)
                        tab[v - f_lo] = (uint32_t)(q + 1);
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int k = 0; k < ITEMS; ++k) {
            const int q = tid + k * BLOCK;
            if (q < m && use_tab) {
                if (q > 0 && lf[q] < lf[q - 1]) bad = true;  // the sorted promise is broken
                const int32_t l = l_r[k];
                int a = l >= f_hi ? m : (l < f_lo ? q + 1 : (int)tab[l - f_lo]);
                a = a < q + 1 ? q + 1 : (a > m ? m : a);
                band[q] = (uint32_t)(a - q - 1);
            } else if (q < m) {
                if (q > 0 && lf[q] < lf[q - 1]) bad = true;  // the sorted promise is broken
                const int32_t l = l_r[k];
                const int32_t f1 = q + 1 < m ? lf[q + 1] : INT32_MAX;
                const int32_t f2 = q + 2 < m ? lf[q + 2] : INT32_MAX;
                const int32_t f3 = q + 3 < m ? lf[q + 3] : INT32_MAX;
                const int32_t f4 = q + 4 < m ? lf[q + 4] : INT32_MAX;
                int a = q + 1 + (f1 <= l) + (f2 <= l) + (f3 <= l) + (f4 <= l);
                if (a == q + 5) {  // first[q + 4] <= l: gallop on
                    int known = q + 4, step = 8, probe = q + 8;  // first[known] <= l
                    while (probe < m && lf[probe] <= l) {
                        known = probe;
                        step <<= 1;
                        probe = q + step;
                    }
                    a = known + 1;
                    int z = probe < m ? probe : m;
                    while (a < z) {
                        const int mid = (a + z) >> 1;
                        if (lf[mid] <= l) a = mid + 1;
                        else z = mid;
                    }
                }
                band[q] = (uint32_t)(a - q - 1);
            }
        }
        __syncthreads();  // first[] is dead: the byte ranges go in its place
        {  // the byte ranges, again every load before any use
            int64_t s_r[ITEMS], o_r[ITEMS];
            const int mc = m > 0 ? m - 1 : 0;
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                const int q = min(tid + k * BLOCK, mc);
                s_r[k] = m > 0 ? size[lo + q] : 1;
                o_r[k] = m > 0 ? off[lo + q] : 0;
            }
#pragma unroll
            for (int k = 0; k < ITEMS; ++k) {
                const int q = tid + k * BLOCK;
                if (q < m) {
                    const int64_t sz = s_r[k], o = o_r[k];
                    if (sz <= 0 || o < 0 || o > INT64_MAX - sz) bad = true;
                    lo64[q] = o;
                    ls64[q] = sz;
                }
            }
        }
        if (!write && __ballot(bad) && (tid & (kWave - 1)) == 0) raise_status(status, MP_EINVAL);
        __syncthreads();
        // band starts: exclusive scan over contiguous chunks
        uint32_t n_pairs;
        {
            const int chunk = (m + BLOCK - 1) / BLOCK;
            const int a0 = min(m, tid * chunk), a1 = min(m, a0 + chunk);
            uint32_t sum = 0;
            for (int i = a0; i < a1; ++i) sum += band[i];
            uint32_t tot;
            uint32_t run = block_exclusive_sum<BLOCK>(sum, &tot, scratch);
            for (int i = a0; i < a1; ++i) {
                const uint32_t v = band[i];
                band[i] = run;
                run += v;
            }
            if (tid == 0) band[m] = tot;
            n_pairs = tot;
        }
        __syncthreads();
        // pairs p in [p_lo, p_hi) of this thread, row-major
        const uint32_t per = (n_pairs + BLOCK - 1) / BLOCK;
        const uint32_t p_lo = min(n_pairs, (uint32_t)tid * per), p_hi = min(n_pairs, p_lo + per);
        int q0 = 0;
        if (p_lo < p_hi) {
            int a = 0, z = m;  // last position whose band starts at or before p_lo
            while (a < z) {
                const int mid = (a + z + 1) >> 1;
                if (band[mid] <= p_lo) a = mid;
                else z = mid - 1;
            }
            q0 = a;
        }
        auto sweep = [&](auto&& on_hit) {
            if (p_lo >= p_hi) return;
            int q = q0;
            uint32_t start = band[q], nxt = band[q + 1];
            int64_t oq = lo64[q], sq = ls64[q];
            for (uint32_t p = p_lo; p < p_hi; ++p) {
                while (nxt <= p) {
                    ++q;
                    start = nxt;
                    nxt = band[q + 1];
                    oq = lo64[q];
                    sq = ls64[q];
                }
                const int j = q + 1 + (int)(p - start);
                if (bytes_meet(oq, sq, lo64[j], ls64[j])) on_hit(q, j);
            }
        };
        uint32_t hits = 0;
        sweep([&](int, int) { ++hits; });
        if (!write) {
            const uint32_t tot = block_reduce<BLOCK>(hits, OpAdd<uint32_t>(), scratch);
            if (tid == 0) segcnt[b] = tot;
        } else {
            uint32_t tot;
            const uint32_t before = block_exclusive_sum<BLOCK>(hits, &tot, scratch);
            int64_t pos = base + before;
            sweep([&](int q, int j) {
                if (pos < cap) {
                    pairs[2 * pos] = lo + q;
                    pairs[2 * pos + 1] = lo + j;
                }
                ++pos;
            });
        }
        __syncthreads();  // LDS is reused by the next trace
    }
}

// One workgroup: exclusive scan of the per-trace counts in place,
// segcnt[n_seg] = total = *n_out; MP_ENOSPC when the total exceeds cap.
__global__ __launch_bounds__(1024) void vb_scan_kernel(int64_t* __restrict__ segcnt, int64_t n_seg,
                                                       int64_t cap, int64_t* __restrict__ n_out,
                                                       int32_t* __restrict__ status) {
    __shared__ uint64_t scratch[1024 / kWave];
    constexpr int kItems = 8;
    uint64_t carry = 0;
    for (int64_t base = 0; base < n_seg; base += 1024 * kItems) {
        const int64_t i0 = base + (int64_t)threadIdx.x * kItems;
        uint64_t v[kItems];
        uint64_t s = 0;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            v[k] = (i0 + k < n_seg) ? (uint64_t)segcnt[i0 + k] : 0;
            s += v[k];
        }
        uint64_t total;
        uint64_t run = carry + block_exclusive_sum<1024>(s, &total, scratch);
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            if (i0 + k < n_seg) segcnt[i0 + k] = (int64_t)run;
            run += v[k];
        }
        carry += total;
    }
    if (threadIdx.x == 0) {
        segcnt[n_seg] = (int64_t)carry;
        *n_out = (int64_t)carry;
        if ((int64_t)carry > cap) raise_status(status, MP_ENOSPC);
    }
}

template <int ITEMS>
hipError_t launch_vb(int write, const int64_t* begin, int64_t n_seg, const int64_t* size,
                     const int32_t* first, const int32_t* last, const int64_t* off, int64_t n,
                     int32_t cap_n, int64_t* segcnt, int64_t* pairs, int64_t cap,
                     int64_t* n_out, int32_t* status, hipStream_t st) {
    auto kern = vb_kernel<kVbBlock, ITEMS>;
    const size_t lds = 20 * (size_t)cap_n + 8;
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    const unsigned grid = (unsigned)(n_seg < 65535 ? n_seg : 65535);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kVbBlock), lds, st, begin, n_seg, size, first, last,
                       off, n, cap_n, segcnt, write, pairs, cap, n_out, status);
    return hipGetLastError();
}

hipError_t launch_vb_any(int write, int items, const int64_t* begin, int64_t n_seg,
                         const int64_t* size, const int32_t* first, const int32_t* last,
                         const int64_t* off, int64_t n, int32_t cap_n, int64_t* segcnt,
                         int64_t* pairs, int64_t cap, int64_t* n_out, int32_t* status,
                         hipStream_t st) {
    switch (items) {
        case 1: return launch_vb<1>(write, begin, n_seg, size, first, last, off, n, cap_n, segcnt, pairs, cap, n_out, status, st);
        case 2: return launch_vb<2>(write, begin, n_seg, size, first, last, off, n, cap_n, segcnt, pairs, cap, n_out, status, st);
        case 4: return launch_vb<4>(write, begin, n_seg, size, first, last, off, n, cap_n, segcnt, pairs, cap, n_out, status, st);
        case 8: return launch_vb<8>(write, begin, n_seg, size, first, last, off, n, cap_n, segcnt, pairs, cap, n_out, status, st);
        default: return hipErrorInvalidValue;
    }
}

struct VLayout {
    size_t flags, segend, reach, cnt, chunk_lo, chunk_tiles, keys0, vals0, keys1, vals1, pf, pl, po, ps, pid,
        pk0, pk1, radix, total;
};

VLayout v_layout(int64_t n, int64_t cap, int64_t n_seg = 1) {
    VLayout L{};
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += (bytes + 255) & ~(size_t)255;
        return at;
    };
    const int64_t nn = n > 0 ? n : 1;
    L.flags = take(sizeof(VFlags));
    L.segend = take(nn * 4);
    L.reach = take(nn * 4);
    const int64_t nc = nn > n_seg ? nn : n_seg;  // also the per-trace counts of a batch
    L.cnt = take((nc + 1) * 8 + scan_workspace_bytes(nc + 1));
    const int64_t ncm = (nn + kChunkRows - 1) / kChunkRows;
    L.chunk_lo = take(ncm * 4);
    L.chunk_tiles = take(ncm * 8 + scan_workspace_bytes(ncm));
    L.keys0 = take(nn * 8);
    L.vals0 = take(nn * 4);
    L.keys1 = take(nn * 8);
    L.vals1 = take(nn * 4);
    L.pf = take(nn * 4);
    L.pl = take(nn * 4);
    L.po = take(nn * 8);
    L.ps = take(nn * 8);
    L.pid = take(nn * 4);
    const int64_t cc = cap > 0 ? cap : 1;
    L.pk0 = take(cc * 8);
    L.pk1 = take(cc * 8);
    const size_t rad_n = radix_workspace_bytes(nn), rad_c = radix_workspace_bytes(cc);
    L.radix = take(rad_n > rad_c ? rad_n : rad_c);
    L.total = o;
    return L;
}

unsigned grid_for(int64_t n, int block, unsigned cap) {
    const int64_t g = (n + block - 1) / block;
    return (unsigned)(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

size_t validate_workspace_bytes(int64_t n, int64_t capacity, int64_t n_seg) {
    return v_layout(n, capacity, n_seg).total;
}

hipError_t launch_validate(const int64_t* begin, int64_t n_seg, const int64_t* size,
                           const int32_t* first, const int32_t* last, const int64_t* off,
                           int64_t n, int64_t max_seg, int64_t* pairs, int64_t cap,
                           int64_t* n_out, bool assume_sorted, void* ws, int32_t* status,
                           hipStream_t st) {
    const VLayout L = v_layout(n, cap, begin ? n_seg : 1);
    if (begin && assume_sorted && max_seg > 0 && max_seg <= MP_BATCH_MAX_TRACE_LEN) {
        // batch of short sorted traces: count per trace, scan, write
        int64_t* segcnt = reinterpret_cast<int64_t*>(static_cast<char*>(ws) + L.cnt);
        int items = 1;
        while (items * kVbBlock < max_seg) items <<= 1;
        hipError_t e = launch_vb_any(0, items, begin, n_seg, size, first, last, off, n,
                                     (int32_t)max_seg, segcnt, pairs, cap, n_out, status, st);
        if (e != hipSuccess) return e;
        if (n_seg <= kVbFuseMax) {
            // short batches: each write-pass workgroup sums the counts before
            // its trace (no scan launch); the last one reports the total
            e = launch_vb_any(2, items, begin, n_seg, size, first, last, off, n, (int32_t)max_seg,
                              segcnt, pairs, cap, n_out, status, st);
        } else {
            hipLaunchKernelGGL(vb_scan_kernel, dim3(1), dim3(1024), 0, st, segcnt, n_seg, cap,
                               n_out, status);
            if (cap > 0)
                e = launch_vb_any(1, items, begin, n_seg, size, first, last, off, n,
                                  (int32_t)max_seg, segcnt, pairs, cap, n_out, status, st);
        }
        if (e != hipSuccess) return e;
        return hipGetLastError();
    }
    char* w = static_cast<char*>(ws);
    VFlags* fl = reinterpret_cast<VFlags*>(w + L.flags);
    int32_t* segend = reinterpret_cast<int32_t*>(w + L.segend);
    int32_t* reach = reinterpret_cast<int32_t*>(w + L.reach);
    int64_t* cnt = reinterpret_cast<int64_t*>(w + L.cnt);
    int64_t* cnt_partial = cnt + (n + 1);
    const int64_t n_chunk_max = (n + kChunkRows - 1) / kChunkRows;
    int32_t* chunk_lo = reinterpret_cast<int32_t*>(w + L.chunk_lo);
    int64_t* chunk_tiles = reinterpret_cast<int64_t*>(w + L.chunk_tiles);
    int64_t* chunk_partial = chunk_tiles + n_chunk_max;
    uint64_t* keys0 = reinterpret_cast<uint64_t*>(w + L.keys0);
    uint32_t* vals0 = reinterpret_cast<uint32_t*>(w + L.vals0);
    uint64_t* keys1 = reinterpret_cast<uint64_t*>(w + L.keys1);
    uint32_t* vals1 = reinterpret_cast<uint32_t*>(w + L.vals1);
    int32_t* pf = reinterpret_cast<int32_t*>(w + L.pf);
    int32_t* pl = reinterpret_cast<int32_t*>(w + L.pl);
    int64_t* po = reinterpret_cast<int64_t*>(w + L.po);
    int64_t* ps = reinterpret_cast<int64_t*>(w + L.ps);
    uint32_t* pid = reinterpret_cast<uint32_t*>(w + L.pid);
    uint64_t* pk0 = reinterpret_cast<uint64_t*>(w + L.pk0);
    uint64_t* pk1 = reinterpret_cast<uint64_t*>(w + L.pk1);
    void* rws = w + L.radix;

    hipLaunchKernelGGL(v_init_kernel, dim3(1), dim3(1), 0, st, fl, n);
    if (n == 0) {
        hipLaunchKernelGGL(v_total_kernel, dim3(1), dim3(1), 0, st, (const int64_t*)&fl->begin1[0],
                           (int64_t)0, cap, n_out, status, (int64_t*)nullptr);
        return hipGetLastError();
    }
    int nbits = 1;  // ids, positions and segment ends are below 2^nbits
    while (nbits < 31 && ((int64_t)1 << nbits) <= n) ++nbits;
    const int64_t* seg = begin ? begin : fl->begin1;
    const int64_t nseg = begin ? n_seg : 1;
    const unsigned g = grid_for(n, kVBlock, 4096);
    if (begin)
        hipLaunchKernelGGL(v_segend_kernel, dim3(grid_for(nseg, 1, 65535)), dim3(256), 0, st, seg,
                           nseg, n, segend, status);
    else
        hipLaunchKernelGGL(v_segend_one_kernel, dim3(g), dim3(kVBlock), 0, st, n, segend);
    hipLaunchKernelGGL(v_check_kernel, dim3(g), dim3(kVBlock), 0, st, size, first, last, off, n,
                       (const int32_t*)segend, fl, status, assume_sorted ? 1 : 0);
    hipError_t e = hipSuccess;
    if (!assume_sorted) {
    // position order for unsorted inputs (every kernel below skips itself otherwise)
    hipLaunchKernelGGL(v_keys_kernel, dim3(g), dim3(kVBlock), 0, st, first, (const int32_t*)segend,
                       n, keys0, vals0, (const VFlags*)fl);
    // a single trace sorts by first alone (bits 0..30); a batch by (segment end, first)
    bool alt = false;
    e = radix_sort_pairs(keys0, vals0, keys1, vals1, n, 0, begin ? 32 + nbits : 31, rws, &alt, st,
                         &fl->sorted);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(v_gather_kernel, dim3(g), dim3(kVBlock), 0, st,
                       (const uint32_t*)(alt ? vals1 : vals0), size, first, last, off, n, pf, pl,
                       po, ps, pid, (const VFlags*)fl);
    }
    // count, scan, write
    hipLaunchKernelGGL(v_rows_kernel, dim3(g), dim3(kVBlock), 0, st, first, last, off, size,
                       (const int32_t*)pf, (const int32_t*)pl, (const int64_t*)po,
                       (const int64_t*)ps, (const uint32_t*)pid, (const int32_t*)segend, n, reach,
                       cnt, keys0, vals0, fl, 0, pairs, cap);
    // long rows in class order: one stable pass over the class byte
    bool calt = false;
    e = radix_sort_pairs(keys0, vals0, keys1, vals1, n, 0, 8, rws, &calt, st);
    if (e != hipSuccess) return e;
    const uint32_t* sorted = calt ? vals1 : vals0;
    hipLaunchKernelGGL(v_chunk_kernel, dim3(grid_for(n_chunk_max, kVBlock / kWave, INT32_MAX)),
                       dim3(kVBlock), 0, st, sorted, n, (const int32_t*)reach, (const VFlags*)fl,
                       n_chunk_max, chunk_lo, chunk_tiles);
    e = device_scan_i64(chunk_tiles, n_chunk_max, true, chunk_partial, nullptr, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(v_tile_kernel, dim3(kTileGrid), dim3(kVBlock), 0, st, first, last, off, size,
                       (const int32_t*)pf, (const int32_t*)pl, (const int64_t*)po,
                       (const int64_t*)ps, (const uint32_t*)pid, (const int32_t*)reach, sorted,
                       (const int32_t*)chunk_lo,
                       (const int64_t*)chunk_tiles, n, (const VFlags*)fl, cnt);
    e = device_scan_i64(cnt, n, false, cnt_partial, nullptr, st);
    if (e != hipSuccess) return e;
    const int64_t tiles = (int64_t)(scan_workspace_bytes(n) / sizeof(int64_t)) - 1;
    hipLaunchKernelGGL(v_total_kernel, dim3(1), dim3(1), 0, st, (const int64_t*)cnt_partial, tiles,
                       cap, n_out, status, cnt + n);
    if (cap > 0) {
        hipLaunchKernelGGL(v_rows_kernel, dim3(g), dim3(kVBlock), 0, st, first, last, off, size,
                           (const int32_t*)pf, (const int32_t*)pl, (const int64_t*)po,
                           (const int64_t*)ps, (const uint32_t*)pid, (const int32_t*)segend, n,
                           reach, cnt, keys0, vals0, fl, 1, pairs, cap);
        hipLaunchKernelGGL(v_long_write_kernel, dim3(kLongGrid), dim3(kVBlock), 0, st, first,
                           last, off, size, (const int32_t*)pf, (const int32_t*)pl,
                           (const int64_t*)po, (const int64_t*)ps, (const uint32_t*)pid,
                           (const int32_t*)reach, (const int64_t*)cnt, sorted, n,
                           (const VFlags*)fl, pairs, cap);
        // unsorted inputs: pairs were written in position order; past the
        // capacity they are replaced by the lexicographically first ones,
        // then sorted by (i, j)
        if (assume_sorted) return hipGetLastError();
        hipLaunchKernelGGL(v_select_kernel, dim3(1), dim3(kSelBlock), 0, st, first, last, off, size,
                           (const int32_t*)pf, (const int32_t*)pl, (const int64_t*)po,
                           (const int64_t*)ps, (const uint32_t*)pid, (const int32_t*)reach,
                           (const int64_t*)cnt, n, (const VFlags*)fl, (const int64_t*)n_out, cap,
                           nbits, pairs);
        const unsigned gc = grid_for(cap, kVBlock, 4096);
        hipLaunchKernelGGL(v_pack_kernel, dim3(gc), dim3(kVBlock), 0, st, (const int64_t*)pairs,
                           (const int64_t*)n_out, cap, nbits, pk0, (const VFlags*)fl);
        bool palt = false;
        e = radix_sort_pairs(pk0, nullptr, pk1, nullptr, cap, 0, 2 * nbits, rws, &palt, st,
                             &fl->sorted);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(v_unpack_kernel, dim3(gc), dim3(kVBlock), 0, st,
                           (const uint64_t*)(palt ? pk1 : pk0), (const int64_t*)n_out, cap, nbits,
                           pairs, (const VFlags*)fl);
    }
    return hipGetLastError();
}

}  // namespace mp
