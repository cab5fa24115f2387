// Wave-level helpers on doubles (gfx950, wave64): one-instruction minimum and DPP wave
// minima.
#pragma once

#include "kr_device.h"
#include "kr_filter.h"

namespace kr {

// Minimum of two non-NaN doubles in one instruction (the compiler's fmin adds operand
// canonicalisation it cannot prove unnecessary here).
__device__ __forceinline__ double vmin(double a, double b)
{
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// One DPP step of a wave minimum over doubles (rows not written keep their own value).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_min_f64(double x)
{
    const uint64_t b = dbits(x);
    const uint32_t lo = (uint32_t)b, hi = (uint32_t)(b >> 32);
    uint32_t ylo, yhi;
    if constexpr (ROWS == 0xF) {  // every lane reads a lane of its own row
        ylo = __builtin_amdgcn_mov_dpp(lo, CTRL, 0xF, 0xF, false);
        yhi = __builtin_amdgcn_mov_dpp(hi, CTRL, 0xF, 0xF, false);
    } else {  // rows outside ROWS keep their own value
        ylo = __builtin_amdgcn_update_dpp(lo, lo, CTRL, ROWS, 0xF, false);
        yhi = __builtin_amdgcn_update_dpp(hi, hi, CTRL, ROWS, 0xF, false);
    }
    return vmin(bitsd(((uint64_t)yhi << 32) | ylo), x);
}

// Minima over the wave of two non-NaN doubles (same DPP pattern as wave_min_u64: pairs,
// quads, half rows, rows, then row broadcasts into rows 1-3), interleaved; results
// uniform.  Every lane must be active.
__device__ __forceinline__ void wave_min2_f64(double &x, double &y)
{
    x = dpp_min_f64<0xB1, 0xF>(x);
    y = dpp_min_f64<0xB1, 0xF>(y);
    x = dpp_min_f64<0x4E, 0xF>(x);
    y = dpp_min_f64<0x4E, 0xF>(y);
    x = dpp_min_f64<0x141, 0xF>(x);
    y = dpp_min_f64<0x141, 0xF>(y);
    x = dpp_min_f64<0x140, 0xF>(x);
    y = dpp_min_f64<0x140, 0xF>(y);
    x = dpp_min_f64<0x142, 0xA>(x);
    y = dpp_min_f64<0x142, 0xA>(y);
    x = dpp_min_f64<0x143, 0xC>(x);
    y = dpp_min_f64<0x143, 0xC>(y);
    x = bitsd(lane_u64(dbits(x), 63));
    y = bitsd(lane_u64(dbits(y), 63));
}

// Position of this lane among the set lanes of m below it.
__device__ __forceinline__ int lane_rank(uint64_t m)
{
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

// ---- shared by the one-wave-per-slab evaluation kernels ------------------------------

typedef __attribute__((address_space(3))) void lds_void;

// Compiler-level ordering of LDS accesses within the wave (the hardware executes one
// wave's LDS instructions in order).
__device__ __forceinline__ void wave_lds_fence()
{
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
}

// s_waitcnt encodings (gfx9): vmcnt [3:0]+[15:14], expcnt [6:4], lgkmcnt [11:8].
#define KR_WAIT_VM0 0x0F70
#define KR_WAIT_LGKM0 0xC07F

// Copy n doubles from global memory into LDS by a one-wave block, W bytes per lane and
// instruction (W = 16 needs n even and both addresses 16-byte aligned).  Lane i of an
// instruction writes LDS bytes [base + W*i, base + W*(i+1)).
template <int W>
__device__ __forceinline__ void copy_to_lds(const double *g, double *l, int n)
{
    const int units = n * 8 / W;
    const int lane = threadIdx.x;
    for (int u0 = 0; u0 < units; u0 += 64) {
        const int u = u0 + lane;
        if (u < units) {
            const void *src = (const char *)g + (size_t)u * W;
            lds_void *dst = (lds_void *)((char *)l + (size_t)u0 * W);
            if constexpr (W == 16)
                __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
            else
                __builtin_amdgcn_global_load_lds(src, dst, 4, 0, 0);
        }
    }
}

__device__ __forceinline__ void emit(const Key &k, int n, double *oT, double *oE, int32_t *oI)
{
    if ((threadIdx.x & 63) == 0) {
        oT[n] = bitsd(k.t);
        oE[n] = bitsd(k.e);
        oI[n] = k.i;
    }
}

// Least (T, E, index) candidate among those with pred(r) true.  Fast path when exactly
// one candidate of the wave qualifies; otherwise a full lexicographic reduction.
template <int R, typename Pred>
__device__ __forceinline__ Key chunk_pick(const double (&vT)[R], const double (&vE)[R], int ibase,
                                          int S, Pred pred)
{
    int cnt = 0;
    Key one = key_none();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const uint64_t m = __ballot(pred(r));
        if (m) {
            cnt += __popcll(m);
            const int L = __ffsll((long long)m) - 1;
            one = Key{lane_u64(dbits(vT[r]), L), lane_u64(dbits(vE[r]), L),
                      lane_i32(ibase, L) + r * S};
        }
    }
    if (cnt == 1) return one;
    Key loc = key_none();
#pragma unroll
    for (int r = 0; r < R; ++r)
        if (pred(r)) {
            const Key c{dbits(vT[r]), dbits(vE[r]), ibase + r * S};
            if (kless(c, loc)) loc = c;
        }
    return wave_min_key(loc);
}

// LDS scratch of the filter: room for `cap` candidates (T, E, index).
struct Scratch {
    double *T, *E;
    int32_t *I;
    int cap;
};

// Frontier of the wave's chunk (invalid slots hold T = E = +inf; valid ones are
// finite); tl, el are each lane's least T and E.  Candidate index of slot r of a lane
// is ibase + r * S.  Writes the frontier in ascending T to o*[0 .. n) and returns n
// (uniform).
//
// A (least in (T, E, index) order) and Z (least in (E, T, index) order) come from wave
// minima and ballots over the slots.  Every other kept point lies strictly inside their box
// (T < T_Z, E < E_A), and only box members can beat a box member, so the box is
// gathered one candidate per lane and each keeps itself iff no other member precedes
// it with energy at or below its own; kept points are placed by their rank in T.  A
// box larger than the scratch takes repeated wave minima instead (same result).
template <int R>
__device__ inline int wave_frontier(const double (&vT)[R], const double (&vE)[R], double tl,
                                    double el, int ibase, int S, const Scratch &sc, double *oT,
                                    double *oE, int32_t *oI)
{
    const int lane = threadIdx.x & 63;
    wave_min2_f64(tl, el);
    const uint64_t tab = dbits(tl), ezb = dbits(el);
    if (tab >= KR_INF_BITS) return 0;  // no valid candidate
    const Key A = chunk_pick<R>(vT, vE, ibase, S, [&](int r) { return dbits(vT[r]) == tab; });
    const double TA = bitsd(A.t), EA = bitsd(A.e), EZ = el;
    const int32_t iA = A.i;
    const bool single = A.e == ezb;  // A has the least energy too: A is Z, nothing beats it
    int nkeep = 0;                   // kept points strictly inside the box
    if (!single) {
        const Key Z = chunk_pick<R>(vT, vE, ibase, S, [&](int r) { return dbits(vE[r]) == ezb; });
        const double TZ = bitsd(Z.t);
        const int32_t iZ = Z.i;
        uint32_t rows = 0;
        int tot = 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const uint64_t m = __ballot(vT[r] < TZ && vE[r] < EA);
            tot += __popcll(m);
            rows |= (m != 0 ? 1u : 0u) << r;
        }
        if (tot > 0 && tot <= sc.cap) {
            int base = 0;
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (rows >> r & 1u) {
                    const bool b = vT[r] < TZ && vE[r] < EA;
                    const uint64_t m = __ballot(b);
                    if (b) {
                        const int q = base + (int)__builtin_amdgcn_mbcnt_hi(
                                                   (uint32_t)(m >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
                        sc.T[q] = vT[r];
                        sc.E[q] = vE[r];
                        sc.I[q] = ibase + r * S;
                    }
                    base += __popcll(m);
                }
            wave_lds_fence();
            const bool mine = lane < tot;
            const int q = min(lane, tot - 1);
            const double xT = sc.T[q], xE = sc.E[q];
            const int32_t xI = sc.I[q];
            bool dom = false;
            for (int y = 0; y < tot; ++y) {
                const double yT = bitsd(lane_u64(dbits(xT), y));
                const double yE = bitsd(lane_u64(dbits(xE), y));
                const int32_t yI = lane_i32(xI, y);
                const bool before = yT < xT || (yT == xT && (yE < xE || (yE == xE && yI < xI)));
                dom = dom || (before && yE <= xE);
            }
            const bool kept = mine && !dom;
            uint64_t km = __ballot(kept);
            nkeep = __popcll(km);
            int rank = 0;  // kept points are strictly ordered in T
            while (km) {
                const int y = __ffsll((long long)km) - 1;
                km &= km - 1;
                rank += bitsd(lane_u64(dbits(xT), y)) < xT ? 1 : 0;
            }
            if (kept) {
                oT[1 + rank] = xT;
                oE[1 + rank] = xE;
                oI[1 + rank] = xI;
            }
            wave_lds_fence();
            if (mine) {  // give the pad rows back
                sc.T[lane] = INFINITY;
                sc.E[lane] = 0.0;
                sc.I[lane] = 0;  // the power pad's upper half holds the indices
            }
        } else if (tot > 0) {
            uint64_t bound = dbits(EA);
            const uint64_t zt = dbits(TZ);
            for (;;) {
                Key loc = key_none();
#pragma unroll
                for (int r = 0; r < R; ++r)
                    if (rows >> r & 1u) {
                        const Key c{dbits(vT[r]), dbits(vE[r]), ibase + r * S};
                        if (c.t < zt && c.e < bound && kless(c, loc)) loc = c;
                    }
                const Key w = wave_min_key(loc);
                if (w.t == KR_INF_BITS) break;
                ++nkeep;
                emit(w, nkeep, oT, oE, oI);
                bound = w.e;
            }
        }
        if (lane == 1) {
            oT[1 + nkeep] = TZ;
            oE[1 + nkeep] = EZ;
            oI[1 + nkeep] = iZ;
        }
    }
    if (lane == 0) {
        oT[0] = TA;
        oE[0] = EA;
        oI[0] = iA;
    }
    return single ? 1 : nkeep + 2;
}

// All-SM column running sums before row i: A0[i], B0[i].  Record N holds the totals;
// record N + 1 is zeros.
struct alignas(16) ColRec {
    double a, b;
};

}  // namespace kr
