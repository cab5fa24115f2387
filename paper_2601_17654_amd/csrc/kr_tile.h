// Exact frontier of one tile of points held by a block (<= KR_BLOCK * CPT points).
//
// The frontier rule: sort by (T, E, idx), keep a point iff its E is strictly below
// every E before it.  The tile first discards points that are provably dominated
// by a point of an earlier time bucket (any point in an earlier bucket has smaller
// T), then sorts only the survivors and scans them.
#pragma once

#include "kr_device.h"

namespace kr {

struct TileLds {
    uint64_t *bkt;  // [nb] bucket minima of E (bit patterns)
    uint64_t *sT;   // [cap] survivors
    uint64_t *sE;
    int32_t *sI;
    int nb;         // power of two, multiple of KR_BLOCK
    int cap;        // >= number of valid points in the tile
};

struct TileScratch {
    uint64_t u64[KR_WAVES];
    int32_t i32[KR_WAVES];
};

// Sort n keys ascending in LDS with a bitonic network whose comparators all put the
// smaller key at the lower index; positions >= n behave as +inf and never move, so n
// need not be a power of two.
__device__ inline void lds_sort_keys(uint64_t *sT, uint64_t *sE, int32_t *sI, int n)
{
    int m = 1;
    while (m < n) m <<= 1;
    for (int k = 2; k <= m; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int q = threadIdx.x; q < (m >> 1); q += KR_BLOCK) {
                int lo, hi;
                if (j == (k >> 1)) {  // first stage of a merge: mirror within the block
                    int blk = q / j, r = q % j;
                    lo = blk * k + r;
                    hi = blk * k + (k - 1 - r);
                } else {
                    lo = 2 * j * (q / j) + (q % j);
                    hi = lo + j;
                }
                if (hi < n) {
                    uint64_t ta = sT[lo], ea = sE[lo], tb = sT[hi], eb = sE[hi];
                    int32_t ia = sI[lo], ib = sI[hi];
                    if (key_less(tb, eb, ib, ta, ea, ia)) {
                        sT[lo] = tb; sE[lo] = eb; sI[lo] = ib;
                        sT[hi] = ta; sE[hi] = ea; sI[hi] = ia;
                    }
                }
            }
            __syncthreads();
        }
    }
}

// vT/vE/vI: this thread's points (slots k with vOk[k]).  Writes the tile frontier in
// ascending T to oT/oE/oI[0 .. count) and returns count (valid in every thread).
template <int CPT>
__device__ inline int tile_frontier(const double (&vT)[CPT], const double (&vE)[CPT],
                                    const int32_t (&vI)[CPT], const bool (&vOk)[CPT],
                                    const TileLds &L, TileScratch &sc, double *oT, double *oE,
                                    int32_t *oI)
{
    // 1. time range of the tile
    uint64_t lo = KR_INF_BITS, hi = 0;
#pragma unroll
    for (int k = 0; k < CPT; ++k)
        if (vOk[k]) {
            uint64_t b = dbits(vT[k]);
            lo = b < lo ? b : lo;
            hi = b > hi ? b : hi;
        }
    lo = block_reduce(lo, (uint64_t)KR_INF_BITS, MinU64(), sc.u64);
    hi = block_reduce(hi, (uint64_t)0, MaxU64(), sc.u64);
    if (lo > hi) return 0;  // empty tile
    const double tlo = bitsd(lo), thi = bitsd(hi);
    const double scale = thi > tlo ? (double)L.nb / (thi - tlo) : 0.0;

    // 2. least E per time bucket (bucket index is monotone in T)
    for (int b = threadIdx.x; b < L.nb; b += KR_BLOCK) L.bkt[b] = KR_INF_BITS;
    __syncthreads();
    int vb[CPT];
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
        vb[k] = 0;
        if (vOk[k]) {
            double x = (vT[k] - tlo) * scale;
            vb[k] = !(x > 0.0) ? 0 : (x < (double)(L.nb - 1) ? (int)x : L.nb - 1);
            atomicMin((unsigned long long *)&L.bkt[vb[k]], (unsigned long long)dbits(vE[k]));
        }
    }
    __syncthreads();

    // 3. exclusive prefix minimum over buckets, in place
    {
        const int per = L.nb / KR_BLOCK;
        const int b0 = threadIdx.x * per;
        uint64_t m = KR_INF_BITS;
        for (int q = 0; q < per; ++q) m = MinU64()(m, L.bkt[b0 + q]);
        uint64_t tot;
        uint64_t pm = block_exclusive(m, (uint64_t)KR_INF_BITS, MinU64(), sc.u64, &tot);
        for (int q = 0; q < per; ++q) {
            uint64_t x = L.bkt[b0 + q];
            L.bkt[b0 + q] = pm;
            pm = MinU64()(pm, x);
        }
    }
    __syncthreads();

    // 4. survivors: E strictly below every earlier bucket's minimum
    bool keep[CPT];
    int nk = 0;
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
        keep[k] = vOk[k] && dbits(vE[k]) < L.bkt[vb[k]];
        nk += keep[k];
    }
    int ns;
    int pos = block_exclusive(nk, 0, SumI32(), sc.i32, &ns);
#pragma unroll
    for (int k = 0; k < CPT; ++k)
        if (keep[k]) {
            L.sT[pos] = dbits(vT[k]);
            L.sE[pos] = dbits(vE[k]);
            L.sI[pos] = vI[k];
            ++pos;
        }
    __syncthreads();

    // 5. exact order of the survivors
    lds_sort_keys(L.sT, L.sE, L.sI, ns);

    // 6. strict prefix-minimum scan and compaction
    const int per = (ns + KR_BLOCK - 1) / KR_BLOCK;
    const int s0 = threadIdx.x * per;
    const int s1 = min(ns, s0 + per);
    uint64_t m = KR_INF_BITS;
    for (int q = s0; q < s1; ++q) m = MinU64()(m, L.sE[q]);
    uint64_t tot;
    const uint64_t best0 = block_exclusive(m, (uint64_t)KR_INF_BITS, MinU64(), sc.u64, &tot);
    uint64_t best = best0;
    int nkeep = 0;
    for (int q = s0; q < s1; ++q) {
        uint64_t e = L.sE[q];
        if (e < best) {
            ++nkeep;
            best = e;
        }
    }
    int count;
    int opos = block_exclusive(nkeep, 0, SumI32(), sc.i32, &count);
    best = best0;
    for (int q = s0; q < s1; ++q) {
        uint64_t e = L.sE[q];
        if (e < best) {
            oT[opos] = bitsd(L.sT[q]);
            oE[opos] = bitsd(e);
            oI[opos] = L.sI[q];
            ++opos;
            best = e;
        }
    }
    __syncthreads();
    return count;
}

}  // namespace kr
