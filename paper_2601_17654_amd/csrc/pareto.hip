// Segmented GetFrontier (Algorithm 1's return value, Algorithm 2's last step).
//
// Rule: within a segment, sort points by (T, E, index) and keep a point iff its E is
// strictly below every E before it -- the non-dominated set, exact duplicates
// resolved to the smallest index.  The rule is decomposable: the frontier of a union
// is the frontier of the union of the parts' frontiers.
//
// Work split: every segment is cut into units (tiles of points, or the frequency
// range of one fused workgroup) whose exact frontiers are written to the unit's slot.
// The union of a segment's unit frontiers is then sorted by a merge sort in LDS and
// scanned: a 256-thread block per segment of up to 512 points, a 1024-thread block
// for the few segments of up to 4096, and beyond that LDS-sized chunks whose
// frontiers are merged pairwise in device memory.  A pairwise merge of two staircases
// needs no sort: an element's rank in the partner comes from a binary search, and it
// survives iff the partner element just before it in key order has a larger E.
#include "kr_filter.h"
#include "kr_launch.h"


namespace kr {

// The layout kernels also clear lists[0], the count of segments that the first merge
// stage passes on (so that the merge needs no launch of its own for it).
__global__ void uniform_layout_kernel(int64_t *seg_off, int64_t *unit_base, int n_seg,
                                      int64_t seg_len, int64_t units_per_seg, int32_t *lists)
{
    const int g = blockIdx.x * KR_BLOCK + threadIdx.x;
    if (g == 0) lists[0] = 0;
    if (g > n_seg) return;
    seg_off[g] = (int64_t)g * seg_len;
    unit_base[g] = (int64_t)g * units_per_seg;
}

hipError_t launch_uniform_layout(int64_t *seg_off, int64_t *unit_base, int n_seg,
                                 int64_t seg_len, int64_t units_per_seg, int32_t *lists,
                                 hipStream_t st)
{
    hipLaunchKernelGGL(uniform_layout_kernel, dim3((n_seg + 1 + KR_BLOCK - 1) / KR_BLOCK),
                       dim3(KR_BLOCK), 0, st, seg_off, unit_base, n_seg, seg_len, units_per_seg,
                       lists);
    return hipGetLastError();
}

// unit_base = exclusive prefix sum of ceil(len_g / tile); one block.
__global__ void __launch_bounds__(KR_BLOCK)
tile_layout_kernel(const int64_t *seg_off, int64_t *unit_base, int n_seg, int tile,
                   int32_t *lists)
{
    __shared__ int64_t sc[KR_WAVES];
    if (threadIdx.x == 0) lists[0] = 0;
    int64_t carry = 0;
    for (int g0 = 0; g0 < n_seg; g0 += KR_BLOCK) {
        const int g = g0 + threadIdx.x;
        int64_t nt = 0;
        if (g < n_seg) {
            const int64_t len = seg_off[g + 1] - seg_off[g];
            nt = len > 0 ? (len + tile - 1) / tile : 0;
        }
        int64_t tot;
        const int64_t ex = block_exclusive(nt, (int64_t)0, SumI64(), sc, &tot);
        if (g < n_seg) unit_base[g] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) unit_base[n_seg] = carry;
}

hipError_t launch_tile_layout(const int64_t *seg_off, int64_t *unit_base, int n_seg, int tile,
                              int32_t *lists, hipStream_t st)
{
    hipLaunchKernelGGL(tile_layout_kernel, dim3(1), dim3(KR_BLOCK), 0, st, seg_off, unit_base,
                       n_seg, tile, lists);
    return hipGetLastError();
}

// Segment holding global unit w (unit_base is non-decreasing).
__device__ __forceinline__ int find_segment(const int64_t *unit_base, int n_seg, int64_t w)
{
    int lo = 0, hi = n_seg - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (unit_base[mid] <= w) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Exact frontier of one tile of up to KR_TILE consecutive points of a segment.  The
// first pass holds KR_SURV_CAP survivors in LDS and defers (count -1) a tile with more;
// the second pass takes only deferred tiles, with LDS for the whole tile, and sorts
// their survivors.
template <bool BIG>
__global__ void __launch_bounds__(KR_BLOCK)
pareto_tile_kernel(const double *T, const double *E, SegLayout L, UnitOut o)
{
    static_assert(KR_TILE == 8 * KR_BLOCK, "a tile is 8 points per thread");
    extern __shared__ double tile_lds[];
    __shared__ FilterShared fsh;
    const int64_t w = blockIdx.x;
    if (w >= L.unit_base[L.n_seg]) return;
    if (BIG && o.cnt[w] >= 0) return;  // done by the first pass
    const int g = find_segment(L.unit_base, L.n_seg, w);
    const int64_t s0 = L.seg_off[g];
    const int64_t start = s0 + (w - L.unit_base[g]) * L.unit_stride;
    const int64_t end = min(start + L.unit_stride, L.seg_off[g + 1]);
    FilterLds fl;
    fl.sh = &fsh;
    fl.sT = (uint64_t *)tile_lds;
    fl.sE = fl.sT + KR_SURV_CAP;
    fl.sI = (int32_t *)(fl.sE + KR_SURV_CAP);
    if (BIG) {
        fl.bT = (uint64_t *)tile_lds;
        fl.bE = fl.bT + KR_TILE;
        fl.bI = (int32_t *)(fl.bE + KR_TILE);
        fl.big_cap = KR_TILE;
    } else {
        fl.defer = true;
    }
    double vT[8], vE[8];
    int32_t vI[8];
    bool ok[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int64_t x = start + threadIdx.x + q * KR_BLOCK;
        ok[q] = x < end;
        // + 0.0 maps -0.0 to +0.0, so that the bit patterns order like the values
        vT[q] = ok[q] ? T[x] + 0.0 : 0.0;
        vE[q] = ok[q] ? E[x] + 0.0 : 0.0;
        vI[q] = (int32_t)(x - s0);
    }
    int parity = 0;
    const int n = tile_frontier<8>(vT, vE, vI, ok, fl, parity, o.T + start, o.E + start,
                                   o.I + start);
    if (threadIdx.x == 0) o.cnt[w] = n;
}

hipError_t launch_pareto_tiles(const double *T, const double *E, const SegLayout &L,
                               int64_t n_units_bound, const UnitOut &o, hipStream_t st)
{
    if (n_units_bound == 0) return hipSuccess;
    const size_t lds = (size_t)KR_SURV_CAP * 20, lds_big = (size_t)KR_TILE * 20;
    hipLaunchKernelGGL(pareto_tile_kernel<false>, dim3((unsigned)n_units_bound), dim3(KR_BLOCK),
                       lds, st, T, E, L, o);
    hipLaunchKernelGGL(pareto_tile_kernel<true>, dim3((unsigned)n_units_bound), dim3(KR_BLOCK),
                       lds_big, st, T, E, L, o);
    return hipGetLastError();
}

// Loads that bypass the CU's L1, for data this block wrote earlier in the same launch.
__device__ __forceinline__ double ld_l2(const double *p)
{
    return bitsd(__hip_atomic_load((const uint64_t *)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ int32_t ld_l2(const int32_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint8_t ld_l2(const uint8_t *p)
{
    const uint32_t word = __hip_atomic_load((const uint32_t *)((uintptr_t)p & ~(uintptr_t)3),
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return (uint8_t)(word >> (8 * ((uintptr_t)p & 3)));
}

// Rank of key (t, e, i) in the sorted staircase b[0..n): number of elements before it.
__device__ __forceinline__ int rank_in(const double *bT, const double *bE, const int32_t *bI,
                                       int n, uint64_t t, uint64_t e, int32_t i)
{
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (key_less(dbits(ld_l2(bT + mid)), dbits(ld_l2(bE + mid)), ld_l2(bI + mid), t, e, i))
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// Merge staircases a = in[sa, sa+na) and b = in[sb, sb+nb) into out[sa ...); returns
// the merged frontier's size.  Every thread of the block must call.
__device__ inline int merge_pair(const PointBufs &in, const PointBufs &out, uint8_t *flags,
                                 int64_t sa, int na, int64_t sb, int nb)
{
    __shared__ int32_t sc[KR_WAVES];
    const double *aT = in.T + sa, *aE = in.E + sa, *bT = in.T + sb, *bE = in.E + sb;
    const int32_t *aI = in.I + sa, *bI = in.I + sb;
    for (int x = threadIdx.x; x < na + nb; x += KR_BLOCK) {
        const bool fromA = x < na;
        const int y = fromA ? x : x - na;
        const double t = ld_l2(fromA ? aT + y : bT + y);
        const double e = ld_l2(fromA ? aE + y : bE + y);
        const int32_t id = ld_l2(fromA ? aI + y : bI + y);
        const int r = fromA ? rank_in(bT, bE, bI, nb, dbits(t), dbits(e), id)
                            : rank_in(aT, aE, aI, na, dbits(t), dbits(e), id);
        const double *oE = fromA ? bE : aE;
        const bool alive = !(r > 0 && ld_l2(oE + r - 1) <= e);
        const int64_t dst = sa + y + r;
        out.T[dst] = t;
        out.E[dst] = e;
        out.I[dst] = id;
        flags[dst] = alive;
    }
    __syncthreads();
    const int n = na + nb;
    int base = 0;
    for (int c0 = 0; c0 < n; c0 += KR_BLOCK) {
        const int x = c0 + threadIdx.x;
        const bool has = x < n;
        double t = 0.0, e = 0.0;
        int32_t id = 0;
        int f = 0;
        if (has) {
            t = ld_l2(out.T + sa + x);
            e = ld_l2(out.E + sa + x);
            id = ld_l2(out.I + sa + x);
            f = ld_l2(flags + sa + x);
        }
        __syncthreads();
        int tot;
        const int pos = block_exclusive(f, 0, SumI32(), sc, &tot);
        if (has && f) {
            out.T[sa + base + pos] = t;
            out.E[sa + base + pos] = e;
            out.I[sa + base + pos] = id;
        }
        base += tot;
        __syncthreads();
    }
    return base;
}

struct FinLds {
    uint64_t sT[KR_FIN_CAP], sE[KR_FIN_CAP];
    int32_t sI[KR_FIN_CAP];
    int32_t upre[KR_FIN_UNITS + 1];
};

// ----------------------------------------------------------------------------
// Union of a segment's unit frontiers -> the segment's frontier in `fin` at the
// segment start, its size in fcnt[g].  `buf` holds the unit slots (free to be
// overwritten once they are gathered).
//
// Segments of at most NT * PER points in at most NT units: one block of NT threads
// per segment sorts the union in LDS by merging.  Thread t gathers points t * PER ..
// t * PER + PER - 1 and sorts them in registers; the sorted runs are then merged
// pairwise, one level per doubling of the run width.  At a level every point finds
// its rank in the partner run by a binary search and moves to (its place in its own
// run) + (that rank) -- keys are distinct, so the places form a permutation.  The
// levels move (T, 16-bit point id) pairs between two buffers; E and the index stay in
// place and are read on a tie in T only.  A strict prefix-minimum scan of E over the
// sorted order gives the frontier.
//
// Three stages: every segment first meets the small instance (a block per segment);
// what it cannot take goes on a list for the large instance (one block per listed
// segment, looping), and what that cannot take on a second list for the chunked
// fallback at the end of this section.
#define KR_FM_SMALL_NT 256
#define KR_FM_SMALL_PER 2
#define KR_FM_LARGE_NT 1024
#define KR_FM_LARGE_PER 4

template <int NT, int PER>
struct MergeLds {
    static constexpr int CAP = NT * PER;
    uint64_t T[2][CAP];
    uint16_t id[2][CAP];
    uint64_t E[CAP];
    int32_t I[CAP];
    int32_t upre[NT + 1];  // upre[u] = points in units before u
    int32_t sc32[NT / 64];
    uint64_t sc64[NT / 64];
};

struct MKey {
    uint64_t t, e;
    int32_t i;
};

__device__ __forceinline__ bool mk_less(const MKey &a, const MKey &b)
{
    return key_less(a.t, a.e, a.i, b.t, b.e, b.i);
}

// Key of the point at a level position (T there, id -> E and index) below another's.
__device__ __forceinline__ bool pos_less(uint64_t ta, int xa, uint64_t tb, int xb,
                                         const uint64_t *E, const int32_t *I)
{
    if (ta != tb) return ta < tb;
    const uint64_t ea = E[xa], eb = E[xb];
    if (ea != eb) return ea < eb;
    return I[xa] < I[xb];
}

// Stage entry: unit prefix of segment g into sh.upre and the point count n, or false
// when the segment has more than NT units or NT * PER points.  Block-uniform.
template <int NT, int PER>
__device__ __forceinline__ bool merge_prefix(int g, const SegLayout &L, const int32_t *ucnt,
                                             MergeLds<NT, PER> &sh, int &n)
{
    const int tid = threadIdx.x;
    const int64_t u0 = L.unit_base[g];
    const int nu = (int)(L.unit_base[g + 1] - u0);
    if (nu > NT) return false;
    const int ex = block_exclusive<int, SumI32, NT / 64>(tid < nu ? ucnt[u0 + tid] : 0, 0,
                                                         SumI32(), sh.sc32, &n);
    if (n > MergeLds<NT, PER>::CAP) return false;
    if (tid < nu) sh.upre[tid] = ex;
    if (tid == 0) sh.upre[nu] = n;
    return true;
}

template <int NT, int PER>
__device__ __forceinline__ void merge_segment(int g, int n, const SegLayout &L,
                                              const PointBufs &buf, const PointBufs &fin,
                                              int32_t *fcnt, MergeLds<NT, PER> &sh)
{
    static_assert(NT * PER <= 65536 && (PER & (PER - 1)) == 0, "16-bit ids, power-of-two runs");
    const int tid = threadIdx.x;
    const int64_t s0 = L.seg_off[g];
    const int nu = (int)(L.unit_base[g + 1] - L.unit_base[g]);
    lds_barrier();  // upre
    const int q0 = min(n, tid * PER), q1 = min(n, q0 + PER);
    MKey k[PER];
    int u = 0;  // unit holding point q0: the last u < nu with upre[u] <= q0
#pragma unroll
    for (int step = NT / 2; step >= 1; step >>= 1)
        if (u + step < nu && sh.upre[u + step] <= q0) u += step;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int x = q0 + j;
        k[j] = MKey{~0ull, ~0ull, 0x7FFFFFFF};  // beyond the segment: sorts last, dropped
        if (x < q1) {
            while (sh.upre[u + 1] <= x) ++u;  // skip ended and empty units (x < upre[nu])
            const int64_t src = s0 + (int64_t)u * L.unit_stride + (x - sh.upre[u]);
            k[j] = MKey{dbits(buf.T[src]), dbits(buf.E[src]), buf.I[src]};
        }
    }
#pragma unroll
    for (int w = 2; w <= PER; w <<= 1)
#pragma unroll
        for (int j = w >> 1; j > 0; j >>= 1)
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int l = i ^ j;
                if (l > i && ((i & w) == 0 ? mk_less(k[l], k[i]) : mk_less(k[i], k[l]))) {
                    const MKey x = k[i];
                    k[i] = k[l];
                    k[l] = x;
                }
            }
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (q0 + j < q1) {
            sh.T[0][q0 + j] = k[j].t;
            sh.id[0][q0 + j] = (uint16_t)(q0 + j);
            sh.E[q0 + j] = k[j].e;
            sh.I[q0 + j] = k[j].i;
        }
    lds_barrier();
    // Sorted runs of width w -> width 2w by merge path: the thread owning output
    // positions [q0, q0 + PER) of a pair of runs (A, then B) finds how many of the first
    // q0 - base outputs come from A (a binary search along that diagonal of the merge),
    // then merges its PER outputs from there, holding the next key of each run.
    int cur = 0;
    for (int w = PER; w < n; w <<= 1) {
        const uint64_t *inT = sh.T[cur];
        const uint16_t *inI = sh.id[cur];
        if (q0 < q1) {
            const int base = q0 & ~(2 * w - 1);
            const int la = min(w, n - base), lb = max(0, min(w, n - base - w));
            const uint64_t *AT = inT + base, *BT = inT + base + w;
            const uint16_t *AI = inI + base, *BI = inI + base + w;
            const int d = q0 - base;
            int lo = max(0, d - lb), hi = min(d, la);
            while (lo < hi) {  // the least i with A[i] after B[d - 1 - i]
                const int mid = (lo + hi) >> 1;
                const int jb = d - 1 - mid;
                if (pos_less(AT[mid], AI[mid], BT[jb], BI[jb], sh.E, sh.I)) lo = mid + 1;
                else hi = mid;
            }
            int i = lo, j = d - lo;
            uint64_t at = i < la ? AT[i] : 0, bt = j < lb ? BT[j] : 0;
            int ai = i < la ? AI[i] : 0, bi = j < lb ? BI[j] : 0;
            uint64_t *const oT = sh.T[cur ^ 1] + q0;
            uint16_t *const oI = sh.id[cur ^ 1] + q0;
            for (int u = 0; u < q1 - q0; ++u) {
                const bool fromA = i < la && (j >= lb || pos_less(at, ai, bt, bi, sh.E, sh.I));
                if (fromA) {
                    oT[u] = at;
                    oI[u] = (uint16_t)ai;
                    ++i;
                    if (i < la) {
                        at = AT[i];
                        ai = AI[i];
                    }
                } else {
                    oT[u] = bt;
                    oI[u] = (uint16_t)bi;
                    ++j;
                    if (j < lb) {
                        bt = BT[j];
                        bi = BI[j];
                    }
                }
            }
        }
        cur ^= 1;
        lds_barrier();
    }
    // keep a point iff its E is below every E before it in key order
    const uint16_t *ord = sh.id[cur];
    uint64_t e[PER];
    uint64_t m = KR_INF_BITS;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        e[j] = q0 + j < q1 ? sh.E[ord[q0 + j]] : KR_INF_BITS;
        m = e[j] < m ? e[j] : m;
    }
    uint64_t all;
    const uint64_t best0 =
        block_exclusive<uint64_t, MinU64, NT / 64>(m, KR_INF_BITS, MinU64(), sh.sc64, &all);
    uint64_t best = best0;
    int nkeep = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (e[j] < best) {
            ++nkeep;
            best = e[j];
        }
    int count;
    int opos = block_exclusive<int, SumI32, NT / 64>(nkeep, 0, SumI32(), sh.sc32, &count);
    best = best0;
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (e[j] < best) {
            const int q = q0 + j;
            fin.T[s0 + opos] = bitsd(sh.T[cur][q]);
            fin.E[s0 + opos] = bitsd(e[j]);
            fin.I[s0 + opos] = sh.I[ord[q]];
            ++opos;
            best = e[j];
        }
    if (tid == 0) fcnt[g] = count;
}

// Stage 1: a block per segment.  lists[0] counts the segments passed on (zero on
// entry), lists[2 ...] holds them; lists[1] (the second list's count) is cleared here.
__global__ void __launch_bounds__(KR_FM_SMALL_NT)
finalize_small_kernel(SegLayout L, PointBufs buf, const int32_t *ucnt, PointBufs fin,
                      int32_t *fcnt, int32_t *lists)
{
    __shared__ MergeLds<KR_FM_SMALL_NT, KR_FM_SMALL_PER> sh;
    const int g = blockIdx.x;
    if (g == 0 && threadIdx.x == 0) lists[1] = 0;
    int n;
    if (merge_prefix(g, L, ucnt, sh, n)) merge_segment(g, n, L, buf, fin, fcnt, sh);
    else if (threadIdx.x == 0) lists[2 + atomicAdd(&lists[0], 1)] = g;
}

// Stage 2: the listed segments, a block each (blocks loop over the list); those it
// cannot take go on the second list (count lists[1], entries from lists[2 + n_seg]).
__global__ void __launch_bounds__(KR_FM_LARGE_NT)
finalize_large_kernel(SegLayout L, PointBufs buf, const int32_t *ucnt, PointBufs fin,
                      int32_t *fcnt, int32_t *lists)
{
    __shared__ MergeLds<KR_FM_LARGE_NT, KR_FM_LARGE_PER> sh;
    const int cnt = lists[0];
    for (int i = blockIdx.x; i < cnt; i += gridDim.x) {
        const int g = lists[2 + i];
        int n;
        if (merge_prefix(g, L, ucnt, sh, n)) merge_segment(g, n, L, buf, fin, fcnt, sh);
        else if (threadIdx.x == 0) lists[2 + L.n_seg + atomicAdd(&lists[1], 1)] = g;
        __syncthreads();  // LDS reuse by the next segment
    }
}

// Stage 3, the segments on the second list: one block per segment (blocks loop over
// the list).  The union is sorted in LDS when it fits; otherwise it is cut into
// LDS-sized chunks whose frontiers are merged pairwise in device memory.
__device__ void finalize_block_segment(int g, const SegLayout &L, const PointBufs &buf,
                                       const int32_t *ucnt, const PointBufs &fin,
                                       int32_t *fcnt, int32_t *runcnt, uint8_t *flags,
                                       FinLds &sh, int32_t *sc)
{
    const int64_t s0 = L.seg_off[g];
    const int64_t u0 = L.unit_base[g];
    const int nu = (int)(L.unit_base[g + 1] - u0);
    // unit sizes and their running offsets
    int64_t total = 0;
    const bool small_units = nu <= KR_FIN_UNITS;
    for (int c0 = 0; c0 < nu; c0 += KR_BLOCK) {
        const int k = c0 + threadIdx.x;
        const int n = k < nu ? ucnt[u0 + k] : 0;
        int tot;
        const int ex = block_exclusive(n, 0, SumI32(), sc, &tot);
        if (small_units && k < nu) sh.upre[k] = (int)total + ex;
        total += tot;
    }
    if (small_units && threadIdx.x == 0) sh.upre[nu] = (int)total;
    __syncthreads();
    if (small_units && total <= KR_FIN_CAP) {
        const int n = (int)total;
        for (int x = threadIdx.x; x < n; x += KR_BLOCK) {
            int lo = 0, hi = nu - 1;  // unit holding element x
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (sh.upre[mid] <= x) lo = mid;
                else hi = mid - 1;
            }
            const int64_t src = s0 + (int64_t)lo * L.unit_stride + (x - sh.upre[lo]);
            sh.sT[x] = dbits(buf.T[src]);
            sh.sE[x] = dbits(buf.E[src]);
            sh.sI[x] = buf.I[src];
        }
        __syncthreads();
        lds_sort_keys(sh.sT, sh.sE, sh.sI, n);
        const int cnt = lds_frontier_scan(sh.sT, sh.sE, sh.sI, n, fin.T + s0, fin.E + s0, fin.I + s0);
        if (threadIdx.x == 0) fcnt[g] = cnt;
        return;
    }
    // Large union: gather contiguously into fin, reduce LDS-sized chunks in place,
    // then merge the chunk staircases pairwise (fin <-> buf).
    int64_t pre = 0;
    for (int k = 0; k < nu; ++k) {
        const int n = ld_l2(ucnt + u0 + k);
        const int64_t src = s0 + (int64_t)k * L.unit_stride;
        for (int x = threadIdx.x; x < n; x += KR_BLOCK) {
            fin.T[s0 + pre + x] = buf.T[src + x];
            fin.E[s0 + pre + x] = buf.E[src + x];
            fin.I[s0 + pre + x] = buf.I[src + x];
        }
        pre += n;
    }
    __syncthreads();
    int32_t *rc = runcnt + s0 / KR_FIN_CAP + g;
    const int nchunks = (int)((total + KR_FIN_CAP - 1) / KR_FIN_CAP);
    for (int c = 0; c < nchunks; ++c) {
        const int64_t c0 = (int64_t)c * KR_FIN_CAP;
        const int n = (int)min((int64_t)KR_FIN_CAP, total - c0);
        for (int x = threadIdx.x; x < n; x += KR_BLOCK) {
            sh.sT[x] = dbits(ld_l2(fin.T + s0 + c0 + x));
            sh.sE[x] = dbits(ld_l2(fin.E + s0 + c0 + x));
            sh.sI[x] = ld_l2(fin.I + s0 + c0 + x);
        }
        __syncthreads();
        lds_sort_keys(sh.sT, sh.sE, sh.sI, n);
        const int cnt = lds_frontier_scan(sh.sT, sh.sE, sh.sI, n, fin.T + s0 + c0, fin.E + s0 + c0,
                                          fin.I + s0 + c0);
        if (threadIdx.x == 0) rc[c] = cnt;
        __syncthreads();
    }
    PointBufs cur = fin, other = buf;
    for (int span = 1; span < nchunks; span <<= 1) {
        for (int r = 0; r < nchunks; r += 2 * span) {
            const int64_t sa = s0 + (int64_t)r * KR_FIN_CAP;
            const int na = ld_l2(rc + r);
            int merged;
            if (r + span < nchunks) {
                const int64_t sb = s0 + (int64_t)(r + span) * KR_FIN_CAP;
                merged = merge_pair(cur, other, flags, sa, na, sb, ld_l2(rc + r + span));
            } else {
                for (int x = threadIdx.x; x < na; x += KR_BLOCK) {
                    other.T[sa + x] = ld_l2(cur.T + sa + x);
                    other.E[sa + x] = ld_l2(cur.E + sa + x);
                    other.I[sa + x] = ld_l2(cur.I + sa + x);
                }
                merged = na;
            }
            __syncthreads();
            if (threadIdx.x == 0) rc[r] = merged;
            __syncthreads();
        }
        const PointBufs t = cur;
        cur = other;
        other = t;
    }
    const int n = nchunks > 0 ? ld_l2(rc) : 0;
    if (cur.T != fin.T) {
        for (int x = threadIdx.x; x < n; x += KR_BLOCK) {
            fin.T[s0 + x] = ld_l2(cur.T + s0 + x);
            fin.E[s0 + x] = ld_l2(cur.E + s0 + x);
            fin.I[s0 + x] = ld_l2(cur.I + s0 + x);
        }
    }
    if (threadIdx.x == 0) fcnt[g] = n;
}

__global__ void __launch_bounds__(KR_BLOCK)
finalize_block_kernel(SegLayout L, PointBufs buf, const int32_t *ucnt, PointBufs fin,
                      int32_t *fcnt, int32_t *runcnt, uint8_t *flags, const int32_t *lists)
{
    __shared__ FinLds sh;
    __shared__ int32_t sc[KR_WAVES];
    const int cnt = lists[1];
    for (int i = blockIdx.x; i < cnt; i += gridDim.x) {
        finalize_block_segment(lists[2 + L.n_seg + i], L, buf, ucnt, fin, fcnt, runcnt, flags,
                               sh, sc);
        __syncthreads();  // LDS reuse by the next segment
    }
}

hipError_t launch_finalize(const SegLayout &L, const PointBufs &buf, const int32_t *ucnt,
                           const PointBufs &fin, int32_t *fcnt, int32_t *runcnt, uint8_t *flags,
                           int32_t *lists, hipStream_t st)
{
    if (L.n_seg == 0) return hipSuccess;
    const dim3 loop_grid(min(L.n_seg, 256));
    hipLaunchKernelGGL(finalize_small_kernel, dim3(L.n_seg), dim3(KR_FM_SMALL_NT), 0, st, L, buf,
                       ucnt, fin, fcnt, lists);
    hipLaunchKernelGGL(finalize_large_kernel, loop_grid, dim3(KR_FM_LARGE_NT), 0, st, L, buf,
                       ucnt, fin, fcnt, lists);
    hipLaunchKernelGGL(finalize_block_kernel, loop_grid, dim3(KR_BLOCK), 0, st, L, buf, ucnt,
                       fin, fcnt, runcnt, flags, lists);
    return hipGetLastError();
}

// out_off = exclusive prefix sum of the per-segment frontier sizes; one block.
__global__ void __launch_bounds__(KR_BLOCK)
count_scan_kernel(int n_seg, const int32_t *fcnt, int64_t *out_off)
{
    __shared__ int64_t sc[KR_WAVES];
    int64_t carry = 0;
    for (int g0 = 0; g0 < n_seg; g0 += KR_BLOCK) {
        const int g = g0 + threadIdx.x;
        const int64_t c = g < n_seg ? fcnt[g] : 0;
        int64_t tot;
        const int64_t ex = block_exclusive(c, (int64_t)0, SumI64(), sc, &tot);
        if (g < n_seg) out_off[g] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) out_off[n_seg] = carry;
}

__global__ void __launch_bounds__(KR_BLOCK)
copy_out_kernel(SegLayout L, PointBufs fin, const int64_t *out_off, int64_t cap,
                int32_t *out_idx, double *out_T, double *out_E)
{
    const int g = blockIdx.x;
    const int64_t dst0 = out_off[g], n = out_off[g + 1] - dst0;
    const int64_t src0 = L.seg_off[g];
    for (int64_t x = threadIdx.x; x < n; x += KR_BLOCK) {
        const int64_t d = dst0 + x;
        if (d >= cap) break;
        out_idx[d] = fin.I[src0 + x];
        out_T[d] = fin.T[src0 + x];
        out_E[d] = fin.E[src0 + x];
    }
}

// Up to KR_OUT_SCAN segments: each block forms its segment's output offset itself (the
// sum of the counts before it, in integers, so equal to the scan's) and copies the
// segment, with no separate scan launch.
#define KR_OUT_SCAN 4096
__global__ void __launch_bounds__(KR_BLOCK)
copy_out_scan_kernel(SegLayout L, PointBufs fin, const int32_t *fcnt, int64_t *out_off,
                     int64_t cap, int32_t *out_idx, double *out_T, double *out_E)
{
    __shared__ int64_t sc[KR_WAVES];
    const int g = blockIdx.x;
    int64_t part = 0;
    for (int h = threadIdx.x; h < g; h += KR_BLOCK) part += fcnt[h];
    const int64_t dst0 = block_reduce(part, (int64_t)0, SumI64(), sc);
    const int64_t n = fcnt[g];
    if (threadIdx.x == 0) {
        out_off[g] = dst0;
        if (g == L.n_seg - 1) out_off[L.n_seg] = dst0 + n;
    }
    const int64_t src0 = L.seg_off[g];
    for (int64_t x = threadIdx.x; x < n; x += KR_BLOCK) {
        const int64_t d = dst0 + x;
        if (d >= cap) break;
        out_idx[d] = fin.I[src0 + x];
        out_T[d] = fin.T[src0 + x];
        out_E[d] = fin.E[src0 + x];
    }
}

hipError_t launch_output(const SegLayout &L, const PointBufs &fin, const int32_t *fcnt,
                         int64_t cap, int64_t *out_off, int32_t *out_idx, double *out_T,
                         double *out_E, hipStream_t st)
{
    if (L.n_seg > 0 && L.n_seg <= KR_OUT_SCAN) {
        hipLaunchKernelGGL(copy_out_scan_kernel, dim3(L.n_seg), dim3(KR_BLOCK), 0, st, L, fin,
                           fcnt, out_off, cap, out_idx, out_T, out_E);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(count_scan_kernel, dim3(1), dim3(KR_BLOCK), 0, st, L.n_seg, fcnt, out_off);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || L.n_seg == 0) return e;
    hipLaunchKernelGGL(copy_out_kernel, dim3(L.n_seg), dim3(KR_BLOCK), 0, st, L, fin, out_off, cap,
                       out_idx, out_T, out_E);
    return hipGetLastError();
}

}  // namespace kr
