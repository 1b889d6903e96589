// The planning strategies that Section 2.3 sets beside greedy_by_size:
// bump_allocation, the baseline that never reuses memory, and the optimum of
// Eq. 2.1, which the thesis reaches through a MIP solver and which here is an
// exhaustive search over placement orders for tiny traces.
#include "internal.hpp"
#include "mp_device.hpp"

namespace mp {

namespace {

constexpr int kSBlock = 256;

// ---------------------------------------------------------------------------
// bump_allocation: each allocation, in the order they happen (first op, then
// id), goes at a running offset that then grows by its size.  Per trace: a
// stable radix sort by (trace, first op), an exclusive scan of the sizes in
// that order, and each offset is its scan value minus its trace's start.

struct BumpFlags {
    uint32_t abort;  // input rejected: every later kernel does nothing
    uint32_t pad;
    unsigned long long sum;
};

__global__ void bump_init_kernel(BumpFlags* fl) {
    fl->abort = 0;
    fl->pad = 0;
    fl->sum = 0;
}

// Checks the tensors (and the trace bounds), and writes each tensor's sort
// key (trace << op_bits) | first with its id.  A grid-stride loop over a
// bounded grid: the blocks add their sums of sizes into one word, and fewer
// blocks mean fewer of those same-address atomics.
__global__ __launch_bounds__(kSBlock) void bump_keys_kernel(
    const int64_t* __restrict__ begin, int64_t n_seg, const int64_t* __restrict__ size,
    const int32_t* __restrict__ first, const int32_t* __restrict__ last, int64_t n,
    int32_t num_ops, int op_bits, uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
    BumpFlags* fl, int32_t* status) {
    __shared__ uint64_t red[kSBlock / kWave];
    const int64_t items = max(n, begin ? n_seg + 1 : (int64_t)0);
    uint32_t bad = 0;
    uint64_t acc = 0;
    for (int64_t i = (int64_t)blockIdx.x * kSBlock + threadIdx.x; i < items;
         i += (int64_t)gridDim.x * kSBlock) {
        if (begin && i <= n_seg) {  // trace bounds: 0 = begin[0] <= ... <= begin[n_seg] = n
            const int64_t b = begin[i];
            if ((i == 0 && b != 0) || (i == n_seg && b != n) || (i < n_seg && begin[i + 1] < b))
                bad = 1;
        }
        if (i < n) {
            const int64_t s = size[i];
            const int32_t f = first[i], l = last[i];
            if (s <= 0 || f < 0 || f > l || l >= num_ops) bad = 1;
            else acc = sat_add(acc, (uint64_t)s);
            int64_t seg = 0;  // the last trace whose begin is <= i
            if (begin) {
                int64_t lo = 0, hi = n_seg - 1;
                while (lo < hi) {
                    const int64_t mid = lo + (hi - lo + 1) / 2;
                    if (begin[mid] <= i) lo = mid;
                    else hi = mid - 1;
                }
                seg = lo;
            }
            keys[i] = ((uint64_t)seg << op_bits) | (uint32_t)max(f, 0);
            vals[i] = (uint32_t)i;
        }
    }
    bad = block_reduce<kSBlock>((uint64_t)bad, OpOr<uint64_t>(), red) != 0;
    acc = block_reduce<kSBlock>(acc, OpSatAdd(), red);
    if (threadIdx.x == 0) {
        if (bad) {
            raise_status(status, MP_EINVAL);
            atomicOr(&fl->abort, 1u);
        }
        const uint64_t old = atomicAdd(&fl->sum, (unsigned long long)acc);
        if (acc > (uint64_t)INT64_MAX || old > (uint64_t)INT64_MAX - acc) {
            raise_status(status, MP_EOVERFLOW);
            atomicOr(&fl->abort, 1u);
        }
    }
}

__global__ __launch_bounds__(kSBlock) void bump_gather_kernel(const int64_t* __restrict__ size,
                                                              const uint32_t* __restrict__ vals,
                                                              int64_t n, int64_t* __restrict__ sz,
                                                              const BumpFlags* fl) {
    if (fl->abort) return;
    const int64_t k = (int64_t)blockIdx.x * kSBlock + threadIdx.x;
    if (k < n) sz[k] = size[vals[k]];
}

// scan[k] = sizes before sorted position k; a trace's tensors hold sorted
// positions [begin[s], begin[s + 1]), so its start is scan[begin[s]].
__global__ __launch_bounds__(kSBlock) void bump_write_kernel(
    const int64_t* __restrict__ begin, int64_t n_seg, const uint64_t* __restrict__ keys,
    const uint32_t* __restrict__ vals, const int64_t* __restrict__ scan,
    const int64_t* __restrict__ total, int64_t n, int op_bits, int64_t* __restrict__ offset_out,
    int64_t* __restrict__ peak_out, const BumpFlags* fl) {
    if (fl->abort) return;
    const int64_t k = (int64_t)blockIdx.x * kSBlock + threadIdx.x;
    auto before = [&](int64_t e) { return e < n ? scan[e] : *total; };
    if (k < n) {
        const int64_t seg = (int64_t)(keys[k] >> op_bits);
        offset_out[vals[k]] = scan[k] - (begin ? before(begin[seg]) : 0);
    }
    const int64_t nseg = begin ? n_seg : 1;
    if (k < nseg)
        peak_out[k] = begin ? before(begin[k + 1]) - before(begin[k]) : *total;
}

struct BumpLayout {
    size_t flags, keys0, keys1, sz, partial, radix, vals0, vals1, end;
};

BumpLayout bump_layout(int64_t n) {
    const size_t nn = (size_t)(n > 0 ? n : 1);
    BumpLayout L;
    size_t at = 0;
    auto take = [&](size_t bytes) {
        const size_t here = at;
        at += (bytes + 255) & ~(size_t)255;
        return here;
    };
    L.flags = take(sizeof(BumpFlags));
    L.keys0 = take(nn * 8);
    L.keys1 = take(nn * 8);
    L.sz = take(nn * 8);
    L.partial = take(scan_workspace_bytes((int64_t)nn));
    L.radix = take(radix_workspace_bytes((int64_t)nn));
    L.vals0 = take(nn * 4);
    L.vals1 = take(nn * 4);
    L.end = at;
    return L;
}

int bit_width64(uint64_t x) { return x ? 64 - __builtin_clzll(x) : 0; }

// ---------------------------------------------------------------------------
// The optimum of Eq. 2.1 for a tiny trace: the least peak over all placement
// orders, each tensor at the lowest offset where it overlaps no placed tensor
// whose lifetime meets its own (sorting an optimal plan by offset gives an
// order that reaches the optimum this way).  One workgroup per trace; each
// thread takes prefixes of the order (unranked from their index) and searches
// below them depth first.  A subtree is cut as soon as its partial peak
// reaches the best peak found so far by any thread of the workgroup, and the
// whole search stops once that best equals the live-bytes lower bound.

constexpr int kOBlock = 256;
constexpr int kOptMaxN = MP_OPT_MAX_N;

struct OptShared {
    int64_t sz[kOptMaxN];
    uint32_t meets[kOptMaxN];  // bit j: lifetimes of i and j meet (j != i)
    // per-thread search state, thread index fastest (no bank conflicts)
    int64_t off[kOptMaxN][kOBlock];
    int64_t peak[kOptMaxN + 1][kOBlock];  // peak after k placements
    uint8_t order[kOptMaxN][kOBlock];     // tensor placed k-th
    uint8_t cand[kOptMaxN + 1][kOBlock];  // next tensor to try at level k
    uint8_t best_order[kOptMaxN][kOBlock];
    unsigned long long best;  // least peak found by the workgroup
    int64_t lb;
    int32_t winner;
    int32_t bad;
};

// Lowest offset for tensor c: 0 or the end of a placed tensor whose lifetime
// meets c's, the least of them where c overlaps none of those tensors.
__device__ int64_t opt_lowest_fit(const OptShared& S, int c, uint32_t placed, int t) {
    const uint32_t nb = placed & S.meets[c];
    const int64_t s = S.sz[c];
    int64_t best = -1;
    for (uint32_t cands = nb | (1u << 31); cands; cands &= cands - 1) {
        const int a = __builtin_ctz(cands);
        const int64_t x = a == 31 ? 0 : S.off[a][t] + S.sz[a];
        if (best >= 0 && x >= best) continue;
        bool free_here = true;
        for (uint32_t m = nb; m && free_here; m &= m - 1) {
            const int j = __builtin_ctz(m);
            const int64_t oj = S.off[j][t];
            if (x < oj + S.sz[j] && oj < x + s) free_here = false;
        }
        if (free_here) best = x;
    }
    return best;
}

__global__ __launch_bounds__(kOBlock) void optimal_kernel(
    const int64_t* __restrict__ begin, const int32_t* __restrict__ num_ops,
    const int64_t* __restrict__ size, const int32_t* __restrict__ first,
    const int32_t* __restrict__ last, int64_t n_tensors, int64_t* __restrict__ offset_out,
    int64_t* __restrict__ peak_out, int32_t* __restrict__ status) {
    __shared__ OptShared S;
    const int t = threadIdx.x;
    const int64_t b0 = begin[blockIdx.x], b1 = begin[blockIdx.x + 1];
    const int64_t nn = b1 - b0;
    if (b0 < 0 || b1 > n_tensors || nn < 0 || nn > kOptMaxN) {
        if (t == 0) raise_status(status, MP_EINVAL);
        return;
    }
    const int n = (int)nn;
    if (t == 0) {
        S.bad = 0;
        S.winner = kOBlock;
    }
    __syncthreads();
    int32_t f = 0, l = 0;
    if (t < n) {
        const int64_t s = size[b0 + t];
        f = first[b0 + t];
        l = last[b0 + t];
        if (s <= 0 || f < 0 || f > l || l >= num_ops[blockIdx.x]) atomicOr(&S.bad, 1);
        S.sz[t] = s;
    }
    __syncthreads();
    if (S.bad) {
        if (t == 0) raise_status(status, MP_EINVAL);
        return;
    }
    // lifetimes that meet, and the live bytes at each tensor's first op (the
    // most live bytes are reached at some tensor's first op)
    __shared__ int32_t sf[kOptMaxN], sl[kOptMaxN];
    if (t < n) {
        sf[t] = f;
        sl[t] = l;
    }
    __syncthreads();
    if (t == 0) {
        uint64_t total = 0;
        int64_t lb = 0;
        for (int i = 0; i < n; ++i) {
            total = sat_add(total, (uint64_t)S.sz[i]);
            uint32_t m = 0;
            int64_t live = 0;
            for (int j = 0; j < n; ++j) {
                if (j != i && sf[i] <= sl[j] && sf[j] <= sl[i]) m |= 1u << j;
                if (sf[j] <= sf[i] && sf[i] <= sl[j]) live += S.sz[j];
            }
            S.meets[i] = m;
            lb = max(lb, live);
        }
        if (total > (uint64_t)INT64_MAX) {
            S.bad = 1;
            raise_status(status, MP_EOVERFLOW);
        }
        S.best = total + 1;  // above any order's peak (at most the sum of sizes)
        S.lb = lb;
    }
    __syncthreads();
    if (S.bad) return;
    if (n == 0) {
        if (t == 0) peak_out[blockIdx.x] = 0;
        return;
    }

    // prefixes: the first d tensors of the order, at least 4 per thread when
    // the trace is large enough
    int d = 0;
    int64_t n_pre = 1;
    while (d < n && n_pre < 4 * kOBlock) n_pre *= n - d++;
    unsigned long long mine = ~0ull;  // this thread's best peak
    for (int64_t p = t; p < n_pre && (int64_t)S.best > S.lb; p += kOBlock) {
        uint32_t placed = 0;
        int64_t q = p, pk = 0;
        bool cut = false;
        for (int k = 0; k < d && !cut; ++k) {  // the p-th prefix, in mixed radix
            const int r = n - k;
            int digit = (int)(q % r);
            q /= r;
            uint32_t free_ids = ((1u << n) - 1u) & ~placed;
            while (digit--) free_ids &= free_ids - 1;
            const int c = __builtin_ctz(free_ids);
            const int64_t x = opt_lowest_fit(S, c, placed, t);
            S.off[c][t] = x;
            S.order[k][t] = (uint8_t)c;
            placed |= 1u << c;
            pk = max(pk, x + S.sz[c]);
            S.peak[k + 1][t] = pk;
            cut = pk >= (int64_t)S.best;
        }
        if (cut) continue;
        int k = d;
        S.cand[k][t] = 0;
        while (k >= d) {
            if (k == n) {  // a complete order
                const unsigned long long v = (unsigned long long)S.peak[n][t];
                if (v < mine) {
                    mine = v;
                    for (int i = 0; i < n; ++i) S.best_order[i][t] = S.order[i][t];
                    atomicMin(&S.best, v);
                }
                --k;
                placed &= ~(1u << S.order[k][t]);
                continue;
            }
            const uint32_t avail = ((1u << n) - 1u) & ~placed & ~((1u << S.cand[k][t]) - 1u);
            if (!avail || (int64_t)S.best <= S.lb) {  // level done: back up
                --k;
                if (k >= d) placed &= ~(1u << S.order[k][t]);
                continue;
            }
            const int c = __builtin_ctz(avail);
            S.cand[k][t] = (uint8_t)(c + 1);
            const int64_t x = opt_lowest_fit(S, c, placed, t);
            const int64_t nk = max(S.peak[k][t], x + S.sz[c]);
            if (nk >= (int64_t)S.best) continue;
            S.off[c][t] = x;
            S.order[k][t] = (uint8_t)c;
            placed |= 1u << c;
            S.peak[k + 1][t] = nk;
            ++k;
            S.cand[k][t] = 0;
        }
    }
    __syncthreads();
    if (mine == S.best) atomicMin(&S.winner, t);
    __syncthreads();
    if (t == S.winner) {  // one optimal plan: the winner's best order, placed again
        uint32_t placed = 0;
        for (int k = 0; k < n; ++k) {
            const int c = S.best_order[k][t];
            const int64_t x = opt_lowest_fit(S, c, placed, t);
            S.off[c][t] = x;
            placed |= 1u << c;
            offset_out[b0 + c] = x;
        }
        peak_out[blockIdx.x] = (int64_t)S.best;
    }
}

}  // namespace

size_t bump_workspace_bytes(int64_t n) {
    if (n < 0 || n >= INT32_MAX) return 0;
    return bump_layout(n).end;
}

hipError_t launch_bump(const int64_t* begin, int64_t n_seg, const int64_t* size,
                       const int32_t* first, const int32_t* last, int64_t n, int32_t num_ops,
                       int64_t* offset_out, int64_t* peak_out, void* ws, int32_t* status,
                       hipStream_t st) {
    const BumpLayout L = bump_layout(n);
    char* w = static_cast<char*>(ws);
    BumpFlags* fl = reinterpret_cast<BumpFlags*>(w + L.flags);
    uint64_t* k0 = reinterpret_cast<uint64_t*>(w + L.keys0);
    uint64_t* k1 = reinterpret_cast<uint64_t*>(w + L.keys1);
    uint32_t* v0 = reinterpret_cast<uint32_t*>(w + L.vals0);
    uint32_t* v1 = reinterpret_cast<uint32_t*>(w + L.vals1);
    int64_t* sz = reinterpret_cast<int64_t*>(w + L.sz);
    int64_t* partial = reinterpret_cast<int64_t*>(w + L.partial);
    const int op_bits = bit_width64(num_ops > 1 ? (uint64_t)(num_ops - 1) : 0);
    const int seg_bits = begin ? bit_width64(n_seg > 1 ? (uint64_t)(n_seg - 1) : 0) : 0;
    const int64_t items = max(n, begin ? n_seg + 1 : (int64_t)0);
    const unsigned nb = (unsigned)((max(items, (int64_t)1) + kSBlock - 1) / kSBlock);
    hipLaunchKernelGGL(bump_init_kernel, dim3(1), dim3(1), 0, st, fl);
    hipLaunchKernelGGL(bump_keys_kernel, dim3(min(nb, 1024u)), dim3(kSBlock), 0, st, begin, n_seg, size,
                       first, last, n, num_ops, op_bits, k0, v0, fl, status);
    bool alt = false;
    hipError_t e = radix_sort_pairs(k0, v0, k1, v1, n, 0, op_bits + seg_bits, w + L.radix, &alt,
                                    st, &fl->abort);
    if (e != hipSuccess) return e;
    const uint64_t* ks = alt ? k1 : k0;
    const uint32_t* vs = alt ? v1 : v0;
    const unsigned ng = (unsigned)((max(n, (int64_t)1) + kSBlock - 1) / kSBlock);
    hipLaunchKernelGGL(bump_gather_kernel, dim3(ng), dim3(kSBlock), 0, st, size, vs, n, sz,
                       (const BumpFlags*)fl);
    if (n > 0) {
        e = device_scan_i64(sz, n, false, partial, nullptr, st, &fl->abort);
        if (e != hipSuccess) return e;
    }
    // the sum of the sizes: the scan's total, or the checked sum (0) when empty
    const int64_t* total = n > 0 ? partial + (scan_workspace_bytes(n) / 8 - 1)
                                 : reinterpret_cast<const int64_t*>(&fl->sum);
    hipLaunchKernelGGL(bump_write_kernel, dim3(nb), dim3(kSBlock), 0, st, begin, n_seg, ks, vs,
                       (const int64_t*)sz, total, n, op_bits, offset_out, peak_out,
                       (const BumpFlags*)fl);
    return hipGetLastError();
}

hipError_t launch_optimal(const int64_t* begin, int64_t n_traces, const int32_t* num_ops,
                          const int64_t* size, const int32_t* first, const int32_t* last,
                          int64_t n_tensors, int64_t* offset_out, int64_t* peak_out,
                          int32_t* status, hipStream_t st) {
    if (n_traces == 0) return hipSuccess;
    hipLaunchKernelGGL(optimal_kernel, dim3((unsigned)n_traces), dim3(kOBlock), 0, st, begin,
                       num_ops, size, first, last, n_tensors, offset_out, peak_out, status);
    return hipGetLastError();
}

}  // namespace mp
