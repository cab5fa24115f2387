// Segmented GetFrontier (Algorithm 1's return value, Algorithm 2's last step).
//
// Rule: within a segment, sort points by (T, E, index) and keep a point iff its E is
// strictly below every E before it -- the non-dominated set, exact duplicates
// resolved to the smallest index.
//
// Work split: every segment is cut into tiles; each tile's exact frontier is found in
// LDS (kr_tile.h).  The frontier rule is decomposable -- the frontier of a union is
// the frontier of the union of the parts' frontiers -- so tile frontiers (strict
// staircases) are merged pairwise, level by level, until one staircase per segment
// remains.  A merge needs no sort: an element's rank in the partner staircase comes
// from a binary search, and it survives iff the partner element just before it in
// key order has a larger E (staircases have strictly falling E).
#include "kr_launch.h"
#include "kr_tile.h"

namespace kr {

__global__ void uniform_layout_kernel(int64_t *seg_off, int64_t *tile_base, int n_seg,
                                      int64_t seg_len, int64_t tiles_per_seg)
{
    const int g = blockIdx.x * KR_BLOCK + threadIdx.x;
    if (g > n_seg) return;
    seg_off[g] = (int64_t)g * seg_len;
    tile_base[g] = (int64_t)g * tiles_per_seg;
}

hipError_t launch_uniform_layout(int64_t *seg_off, int64_t *tile_base, int n_seg,
                                 int64_t seg_len, int64_t tiles_per_seg, hipStream_t st)
{
    hipLaunchKernelGGL(uniform_layout_kernel, dim3((n_seg + 1 + KR_BLOCK - 1) / KR_BLOCK),
                       dim3(KR_BLOCK), 0, st, seg_off, tile_base, n_seg, seg_len, tiles_per_seg);
    return hipGetLastError();
}

// tile_base = exclusive prefix sum of ceil(len_g / tile); one block.
__global__ void __launch_bounds__(KR_BLOCK)
tile_layout_kernel(const int64_t *seg_off, int64_t *tile_base, int n_seg, int tile)
{
    __shared__ int64_t sc[KR_WAVES];
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
        if (g < n_seg) tile_base[g] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) tile_base[n_seg] = carry;
}

hipError_t launch_tile_layout(const int64_t *seg_off, int64_t *tile_base, int n_seg, int tile,
                              hipStream_t st)
{
    hipLaunchKernelGGL(tile_layout_kernel, dim3(1), dim3(KR_BLOCK), 0, st, seg_off, tile_base,
                       n_seg, tile);
    return hipGetLastError();
}

__device__ __forceinline__ int64_t tile_start(const SegLayout &L, int64_t k)
{
    return (k / L.tiles_per_group) * L.group_elems + (k % L.tiles_per_group) * (int64_t)L.tile;
}

// Segment holding global tile w (tile_base is non-decreasing).
__device__ __forceinline__ int find_segment(const int64_t *tile_base, int n_seg, int64_t w)
{
    int lo = 0, hi = n_seg - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tile_base[mid] <= w) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

template <int CPT>
__global__ void __launch_bounds__(KR_BLOCK)
pareto_tile_kernel(const double *T, const double *E, SegLayout L, TileOut o)
{
    extern __shared__ uint64_t tile_lds[];
    __shared__ TileScratch sc;
    const int64_t w = blockIdx.x;
    if (w >= L.tile_base[L.n_seg]) return;
    const int g = find_segment(L.tile_base, L.n_seg, w);
    const int64_t k = w - L.tile_base[g];
    const int64_t s0 = L.seg_off[g];
    const int64_t start = s0 + k * L.tile;
    const int64_t end = min(start + (int64_t)L.tile, L.seg_off[g + 1]);
    TileLds tl;
    tl.nb = o.nb;
    tl.cap = L.tile;
    tl.bkt = tile_lds;
    tl.sT = tl.bkt + o.nb;
    tl.sE = tl.sT + L.tile;
    tl.sI = (int32_t *)(tl.sE + L.tile);
    double vT[CPT], vE[CPT];
    int32_t vI[CPT];
    bool ok[CPT];
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        const int64_t x = start + threadIdx.x + q * KR_BLOCK;
        ok[q] = x < end;
        vT[q] = ok[q] ? T[x] : 0.0;
        vE[q] = ok[q] ? E[x] : 0.0;
        vI[q] = (int32_t)(x - s0);
    }
    const int n = tile_frontier<CPT>(vT, vE, vI, ok, tl, sc, o.T + start, o.E + start, o.I + start);
    if (threadIdx.x == 0) o.cnt[w] = n;
}

hipError_t launch_pareto_tiles(const double *T, const double *E, const SegLayout &L,
                               int64_t n_tiles_bound, const TileOut &o, int cpt, hipStream_t st)
{
    if (n_tiles_bound == 0) return hipSuccess;
    const size_t lds = (size_t)o.nb * 8 + (size_t)L.tile * 20;
    const dim3 grid((unsigned)n_tiles_bound), block(KR_BLOCK);
    if (cpt == 8) hipLaunchKernelGGL(pareto_tile_kernel<8>, grid, block, lds, st, T, E, L, o);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// Number of elements of staircase (bT, bE, bI)[0..n) that precede key (t, e, i).
__device__ __forceinline__ int rank_in(const double *bT, const double *bE, const int32_t *bI,
                                       int n, uint64_t t, uint64_t e, int32_t i)
{
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (key_less(dbits(bT[mid]), dbits(bE[mid]), bI[mid], t, e, i)) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__global__ void __launch_bounds__(KR_BLOCK)
merge_kernel(SegLayout L, int level, int64_t pairs_per_seg, PointBufs in, const int32_t *cnt_in,
             PointBufs out, int32_t *cnt_out, uint8_t *flags)
{
    __shared__ int32_t sc[KR_WAVES];
    const int64_t w = blockIdx.x;
    const int g = (int)(w / pairs_per_seg);
    const int64_t q = w % pairs_per_seg;
    if (g >= L.n_seg) return;
    const int64_t tb = L.tile_base[g];
    const int64_t nt = L.tile_base[g + 1] - tb;
    const int64_t kA = q << (level + 1);
    if (kA >= nt) return;
    const int64_t kB = kA + ((int64_t)1 << level);
    const int64_t sA = L.seg_off[g] + tile_start(L, kA);
    const int nA = cnt_in[tb + kA];
    if (kB >= nt) {  // no partner: carry the staircase over
        for (int x = threadIdx.x; x < nA; x += KR_BLOCK) {
            out.T[sA + x] = in.T[sA + x];
            out.E[sA + x] = in.E[sA + x];
            out.I[sA + x] = in.I[sA + x];
        }
        if (threadIdx.x == 0) cnt_out[tb + kA] = nA;
        return;
    }
    const int64_t sB = L.seg_off[g] + tile_start(L, kB);
    const int nB = cnt_in[tb + kB];
    const double *aT = in.T + sA, *aE = in.E + sA, *bT = in.T + sB, *bE = in.E + sB;
    const int32_t *aI = in.I + sA, *bI = in.I + sB;
    // merged order, with a survival flag per element
    for (int x = threadIdx.x; x < nA + nB; x += KR_BLOCK) {
        const bool fromA = x < nA;
        const int y = fromA ? x : x - nA;
        const double t = fromA ? aT[y] : bT[y];
        const double e = fromA ? aE[y] : bE[y];
        const int32_t id = fromA ? aI[y] : bI[y];
        const int r = fromA ? rank_in(bT, bE, bI, nB, dbits(t), dbits(e), id)
                            : rank_in(aT, aE, aI, nA, dbits(t), dbits(e), id);
        const double *oE = fromA ? bE : aE;
        const bool alive = !(r > 0 && oE[r - 1] <= e);
        const int64_t dst = sA + y + r;
        out.T[dst] = t;
        out.E[dst] = e;
        out.I[dst] = id;
        flags[dst] = alive;
    }
    __syncthreads();
    // stable in-place compaction of the survivors
    const int n = nA + nB;
    int base = 0;
    for (int c0 = 0; c0 < n; c0 += KR_BLOCK) {
        const int x = c0 + threadIdx.x;
        const bool has = x < n;
        double t = 0.0, e = 0.0;
        int32_t id = 0;
        int f = 0;
        if (has) {
            t = out.T[sA + x];
            e = out.E[sA + x];
            id = out.I[sA + x];
            f = flags[sA + x];
        }
        __syncthreads();
        int tot;
        const int pos = block_exclusive(f, 0, SumI32(), sc, &tot);
        if (has && f) {
            out.T[sA + base + pos] = t;
            out.E[sA + base + pos] = e;
            out.I[sA + base + pos] = id;
        }
        base += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) cnt_out[tb + kA] = base;
}

hipError_t launch_merge_level(const SegLayout &L, int level, int64_t max_tiles,
                              const PointBufs &in, const int32_t *cnt_in, const PointBufs &out,
                              int32_t *cnt_out, uint8_t *flags, hipStream_t st)
{
    const int64_t span = (int64_t)1 << (level + 1);
    const int64_t pairs = (max_tiles + span - 1) / span;
    const int64_t blocks = pairs * L.n_seg;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(merge_kernel, dim3((unsigned)blocks), dim3(KR_BLOCK), 0, st, L, level,
                       pairs, in, cnt_in, out, cnt_out, flags);
    return hipGetLastError();
}

// out_off = exclusive prefix sum of the per-segment frontier sizes; one block.
__global__ void __launch_bounds__(KR_BLOCK)
count_scan_kernel(SegLayout L, const int32_t *cnt, int64_t *out_off)
{
    __shared__ int64_t sc[KR_WAVES];
    int64_t carry = 0;
    for (int g0 = 0; g0 < L.n_seg; g0 += KR_BLOCK) {
        const int g = g0 + threadIdx.x;
        int64_t c = 0;
        if (g < L.n_seg && L.tile_base[g + 1] > L.tile_base[g]) c = cnt[L.tile_base[g]];
        int64_t tot;
        const int64_t ex = block_exclusive(c, (int64_t)0, SumI64(), sc, &tot);
        if (g < L.n_seg) out_off[g] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) out_off[L.n_seg] = carry;
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

hipError_t launch_finish(const SegLayout &L, const PointBufs &fin, const int32_t *cnt,
                         int64_t cap, int64_t *out_off, int32_t *out_idx, double *out_T,
                         double *out_E, hipStream_t st)
{
    hipLaunchKernelGGL(count_scan_kernel, dim3(1), dim3(KR_BLOCK), 0, st, L, cnt, out_off);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || L.n_seg == 0) return e;
    hipLaunchKernelGGL(copy_out_kernel, dim3(L.n_seg), dim3(KR_BLOCK), 0, st, L, fin, out_off, cap,
                       out_idx, out_T, out_E);
    return hipGetLastError();
}

}  // namespace kr
