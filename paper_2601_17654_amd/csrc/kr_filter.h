// Exact frontier of a tile of points held in registers by a block.
//
// Frontier rule (GetFrontier): in (T, E, index) order keep a point iff its E is
// strictly below every E before it.  Equivalently, the frontier is produced by
// repeated lexicographic minima: the first point is the (T, E, index)-minimum of the
// tile; each next point is the minimum among the points whose E is below the last
// point's E.  A tile of candidates of one frequency has a frontier of only a few
// points and few candidates beat the first point's energy, so the tile is reduced to
// those survivors with one block-wide minimum and one ballot compaction; a single
// wave finishes them.  If there are too many survivors the block repeats the
// block-wide minimum instead (no capacity limit, same result).
#pragma once

#include "kr_device.h"

#define KR_SURV_CAP 256

namespace kr {

struct Key {
    uint64_t t, e;  // bit patterns of T, E (non-negative doubles order like integers)
    int32_t i;
};

__device__ __forceinline__ Key key_none() { return Key{KR_INF_BITS, KR_INF_BITS, 0x7FFFFFFF}; }
__device__ __forceinline__ bool kless(const Key &a, const Key &b)
{
    return key_less(a.t, a.e, a.i, b.t, b.e, b.i);
}

__device__ __forceinline__ int32_t wave_min_i32(int32_t x)
{
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const int32_t y = __shfl_xor(x, d, 64);
        x = y < x ? y : x;
    }
    return x;
}

// Lexicographic minimum over the wave (all lanes active; result uniform).  Ties on T
// are resolved by E, then by index, only when they occur.
__device__ inline Key wave_min_key(const Key &k)
{
    const uint64_t tm = wave_min_u64(k.t);
    const bool ht = k.t == tm;
    uint64_t m = __ballot(ht);
    if (__popcll(m) == 1) {
        const int lane = __ffsll((long long)m) - 1;
        return Key{tm, lane_u64(k.e, lane), lane_i32(k.i, lane)};
    }
    const uint64_t em = wave_min_u64(ht ? k.e : KR_INF_BITS);
    const bool he = ht && k.e == em;
    m = __ballot(he);
    if (__popcll(m) == 1) {
        const int lane = __ffsll((long long)m) - 1;
        return Key{tm, em, lane_i32(k.i, lane)};
    }
    return Key{tm, em, wave_min_i32(he ? k.i : 0x7FFFFFFF)};
}

struct FilterShared {
    Key slot[2][KR_WAVES];
    int32_t wtot[2][KR_WAVES];
    int32_t nemit;
};

struct FilterLds {
    FilterShared *sh;
    uint64_t *sT, *sE;  // [KR_SURV_CAP] survivors
    int32_t *sI;
    // Optional room for big_cap survivors, sorted there when more than KR_SURV_CAP beat
    // the first point; with none, `defer` returns -1 for such a tile instead of taking
    // one block-wide minimum per kept point.
    uint64_t *bT = nullptr, *bE = nullptr;
    int32_t *bI = nullptr;
    int big_cap = 0;
    bool defer = false;
};

// Block-wide lexicographic minimum (one barrier; the two slot sets alternate so
// back-to-back calls need no second barrier).  The barriers of this file order LDS
// traffic only; the tile's outputs are not read back by the block.
__device__ inline Key block_min_key(const Key &k, FilterShared *sh, int &parity)
{
    const Key w = wave_min_key(k);
    Key *slot = sh->slot[parity];
    parity ^= 1;
    if ((threadIdx.x & 63) == 0) slot[threadIdx.x >> 6] = w;
    lds_barrier();
    Key b = slot[0];
#pragma unroll
    for (int q = 1; q < KR_WAVES; ++q) {
        const Key o = slot[q];
        if (kless(o, b)) b = o;
    }
    return b;
}

__device__ inline void lds_sort_keys(uint64_t *sT, uint64_t *sE, int32_t *sI, int n);
__device__ inline int lds_frontier_scan(const uint64_t *sT, const uint64_t *sE, const int32_t *sI,
                                        int n, double *oT, double *oE, int32_t *oI);

// Frontier of the block's points (slots k < CAP with ok[k]) written in ascending T to
// oT/oE/oI[0 .. n); returns n in every thread (-1 for a tile deferred as described in
// FilterLds).  Every thread of the block must call.
template <int CAP>
__device__ inline int tile_frontier(const double (&vT)[CAP], const double (&vE)[CAP],
                                    const int32_t (&vI)[CAP], const bool (&ok)[CAP],
                                    const FilterLds &L, int &parity, double *oT, double *oE,
                                    int32_t *oI)
{
    Key loc = key_none();
#pragma unroll
    for (int k = 0; k < CAP; ++k)
        if (ok[k]) {
            const Key c{dbits(vT[k]), dbits(vE[k]), vI[k]};
            if (kless(c, loc)) loc = c;
        }
    const Key A = block_min_key(loc, L.sh, parity);
    if (A.t == KR_INF_BITS) return 0;
    if (threadIdx.x == 0) {
        oT[0] = bitsd(A.t);
        oE[0] = bitsd(A.e);
        oI[0] = A.i;
    }
    // candidates below the first point's energy; everything else it dominates
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t below = ((uint64_t)1 << lane) - 1;
    int wcount = 0;
#pragma unroll
    for (int k = 0; k < CAP; ++k) wcount += __popcll(__ballot(ok[k] && dbits(vE[k]) < A.e));
    int32_t *wt = L.sh->wtot[parity];
    parity ^= 1;
    if (lane == 0) wt[wave] = wcount;
    lds_barrier();
    int base = 0, total = 0;
#pragma unroll
    for (int q = 0; q < KR_WAVES; ++q) {
        const int x = wt[q];
        base += q < wave ? x : 0;
        total += x;
    }
    if (total == 0) return 1;
    if (total <= KR_SURV_CAP) {
#pragma unroll
        for (int k = 0; k < CAP; ++k) {
            const bool sv = ok[k] && dbits(vE[k]) < A.e;
            const uint64_t m = __ballot(sv);
            if (sv) {
                const int pos = base + __popcll(m & below);
                L.sT[pos] = dbits(vT[k]);
                L.sE[pos] = dbits(vE[k]);
                L.sI[pos] = vI[k];
            }
            base += __popcll(m);
        }
        lds_barrier();
        if (wave == 0) {
            uint64_t bound = A.e;
            int n = 1;
            for (;;) {
                Key c = key_none();
                for (int x = lane; x < total; x += 64) {
                    const Key it{L.sT[x], L.sE[x], L.sI[x]};
                    if (it.e < bound && kless(it, c)) c = it;
                }
                const Key w = wave_min_key(c);
                if (w.t == KR_INF_BITS) break;
                if (lane == 0) {
                    oT[n] = bitsd(w.t);
                    oE[n] = bitsd(w.e);
                    oI[n] = w.i;
                }
                ++n;
                bound = w.e;
            }
            if (lane == 0) L.sh->nemit = n;
        }
        lds_barrier();
        return L.sh->nemit;
    }
    if (total <= L.big_cap) {
        // Many survivors: sort them in (T, E, index) order and keep each one whose E is
        // below every earlier survivor's.  Points that are not survivors have E at or
        // above A's and A precedes them all, so they can neither be kept nor matter.
#pragma unroll
        for (int k = 0; k < CAP; ++k) {
            const bool sv = ok[k] && dbits(vE[k]) < A.e;
            const uint64_t m = __ballot(sv);
            if (sv) {
                const int pos = base + __popcll(m & below);
                L.bT[pos] = dbits(vT[k]);
                L.bE[pos] = dbits(vE[k]);
                L.bI[pos] = vI[k];
            }
            base += __popcll(m);
        }
        __syncthreads();
        lds_sort_keys(L.bT, L.bE, L.bI, total);
        return 1 + lds_frontier_scan(L.bT, L.bE, L.bI, total, oT + 1, oE + 1, oI + 1);
    }
    if (L.defer) return -1;
    // many survivors: repeat the block-wide minimum over the registers
    uint64_t bound = A.e;
    int n = 1;
    for (;;) {
        Key c = key_none();
#pragma unroll
        for (int k = 0; k < CAP; ++k)
            if (ok[k] && dbits(vE[k]) < bound) {
                const Key x{dbits(vT[k]), dbits(vE[k]), vI[k]};
                if (kless(x, c)) c = x;
            }
        const Key B = block_min_key(c, L.sh, parity);
        if (B.t == KR_INF_BITS) break;
        if (threadIdx.x == 0) {
            oT[n] = bitsd(B.t);
            oE[n] = bitsd(B.e);
            oI[n] = B.i;
        }
        ++n;
        bound = B.e;
    }
    return n;
}

// Sort n keys ascending in LDS with a bitonic network whose comparators all put the
// smaller key at the lower index; positions >= n behave as +inf and never move, so n
// need not be a power of two.  Every thread of the block must call.
__device__ inline void lds_sort_keys(uint64_t *sT, uint64_t *sE, int32_t *sI, int n)
{
    int m = 1, lm = 0;
    while (m < n) {
        m <<= 1;
        ++lm;
    }
    for (int lk = 1; lk <= lm; ++lk) {
        const int k = 1 << lk;
        for (int lj = lk - 1; lj >= 0; --lj) {
            const int j = 1 << lj;  // q / j and q % j by shift and mask
            for (int q = threadIdx.x; q < (m >> 1); q += KR_BLOCK) {
                int lo, hi;
                if (lj == lk - 1) {  // first stage of a merge: mirror within the block
                    const int blk = q >> lj, r = q & (j - 1);
                    lo = blk * k + r;
                    hi = blk * k + (k - 1 - r);
                } else {
                    lo = ((q >> lj) << (lj + 1)) + (q & (j - 1));
                    hi = lo + j;
                }
                if (hi < n) {
                    const uint64_t ta = sT[lo], ea = sE[lo], tb = sT[hi], eb = sE[hi];
                    const int32_t ia = sI[lo], ib = sI[hi];
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

// Strict prefix-minimum scan of n sorted keys in LDS: keeps a key iff its E is below
// every earlier E; writes the kept keys in order to oT/oE/oI and returns their count
// (every thread).  Every thread of the block must call.
__device__ inline int lds_frontier_scan(const uint64_t *sT, const uint64_t *sE, const int32_t *sI,
                                        int n, double *oT, double *oE, int32_t *oI)
{
    __shared__ uint64_t sc64[KR_WAVES];
    __shared__ int32_t sc32[KR_WAVES];
    const int per = (n + KR_BLOCK - 1) / KR_BLOCK;
    const int s0 = threadIdx.x * per;
    const int s1 = min(n, s0 + per);
    uint64_t m = KR_INF_BITS;
    for (int q = s0; q < s1; ++q) m = MinU64()(m, sE[q]);
    uint64_t tot;
    const uint64_t best0 = block_exclusive(m, (uint64_t)KR_INF_BITS, MinU64(), sc64, &tot);
    uint64_t best = best0;
    int nkeep = 0;
    for (int q = s0; q < s1; ++q)
        if (sE[q] < best) {
            ++nkeep;
            best = sE[q];
        }
    int count;
    int opos = block_exclusive(nkeep, 0, SumI32(), sc32, &count);
    best = best0;
    for (int q = s0; q < s1; ++q) {
        const uint64_t e = sE[q];
        if (e < best) {
            oT[opos] = bitsd(sT[q]);
            oE[opos] = bitsd(e);
            oI[opos] = sI[q];
            ++opos;
            best = e;
        }
    }
    return count;
}

}  // namespace kr
