// Launch-timing frontier of two operation sequences (Appendix B's dynamic program), one
// instance per 64-lane workgroup.
//
// The cells P(i, j) (suffixes from S1[i] and S2[j]) are filled from (I, J) back to
// (0, 0), row by row, so every successor is ready.  Per cell:
//   * one lane per decision slot (S1 op alone, S2 op alone, S1's communication
//     overlapped with k of S2's computations, the same swapped) prices its group with
//     the fluid overlap walk and checks that it is allowed; the allowed slots, in that
//     order, become the cell's sources;
//   * the candidates are (group + successor point) over the sources, in source order
//     and then the successor's order; their index is their generation order;
//   * a candidate is kept iff no candidate before it in (T, E, index) order has energy at
//     or below its own (GetFrontier with exact duplicates to the first), decided by
//     comparing against every candidate (cells hold tens of candidates, so this beats
//     sorting): with at most 64 candidates one per lane, through lane reads; otherwise
//     through LDS broadcast reads; a kept point's rank is the number of kept points
//     with a smaller time;
//   * the kept points go to an LDS arena with their back-pointer (source, point).
// The schedules of P(0, 0) are then walked back one lane per point.
#include <math.h>

#include "kr_device.h"
#include "kr_launch.h"

namespace kr {

namespace {

constexpr int kSlots = 2 + 2 * KR_DP_MAX_K;

// Value of lane `src` (per-lane index) for a 64-bit quantity.
__device__ __forceinline__ uint64_t shfl_u64(uint64_t x, int src)
{
    const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)x, src, 64);
    const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(x >> 32), src, 64);
    return ((uint64_t)hi << 32) | lo;
}

// An instance is one wave, whose LDS accesses execute in order: ordering them for the
// compiler is all the synchronisation a cell needs.
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

__device__ __forceinline__ void dp_alone(const double *op, double ps, double *T, double *E)
{
    const double t = op[0], p = op[1];
    *T = t;
    *E = t * p + ps * t;
}

// A communication `c` with the computations ops[r0], ops[r0 + 1], ... ops[r0 + k - 1].
__device__ __forceinline__ void dp_group(const double *ops, int c, int r0, int k, double ps,
                                         double *T, double *E)
{
    const double tc = ops[4 * c], pc = ops[4 * c + 1];
    double tau = 0.0, e = 0.0;
    for (int r = 0; r < k; ++r) {
        const double *o = ops + 4 * (r0 + r);
        const double t0 = o[0], p0 = o[1], t1 = o[2], p1 = o[3];
        if (tau < tc) {
            const double nt = tau + t1;
            if (nt <= tc) {
                e = e + t1 * p1;
                tau = nt;
            } else {
                const double dt = tc - tau;
                const double rem = 1.0 - dt / t1;
                const double ta = rem * t0;
                e = e + dt * p1;
                e = e + ta * p0;
                tau = tc + ta;
            }
        } else {
            e = e + t0 * p0;
            tau = tau + t0;
        }
    }
    const double t = tau > tc ? tau : tc;
    *T = t;
    *E = (e + tc * pc) + ps * t;
}

struct Slots {
    int va, vb, nc, nd;  // allowed: S1 alone, S2 alone, overlaps of each kind
};

__device__ __forceinline__ Slots dp_slots(const DpArgs &a, int i, int j)
{
    Slots s;
    s.va = i < a.I;
    s.vb = j < a.J;
    s.nc = i < a.I && a.kind[i] == 1 ? min(a.kmax, (int)a.run2[j]) : 0;
    s.nd = j < a.J && a.kind[a.I + j] == 1 ? min(a.kmax, (int)a.run1[i]) : 0;
    return s;
}

// Source r of cell (i, j) -> decision code (case * 32 + k) and successor cell.
__device__ __forceinline__ int dp_decode(const DpArgs &a, int i, int j, int r, int *ni, int *nj)
{
    const Slots s = dp_slots(a, i, j);
    if (r < s.va) {
        *ni = i + 1;
        *nj = j;
        return 0;
    }
    r -= s.va;
    if (r < s.vb) {
        *ni = i;
        *nj = j + 1;
        return 32;
    }
    r -= s.vb;
    if (r < s.nc) {
        *ni = i + 1;
        *nj = j + r + 1;
        return 64 + r + 1;
    }
    r -= s.nc;
    *ni = i + r + 1;
    *nj = j + 1;
    return 96 + r + 1;
}

// Byte offsets of the LDS sections of one instance (all 8-byte aligned).
struct DpLds {
    int ops, arT, arE, cT, cE, sT, sE, soff, sstart, arB, cstart, ccnt, csrc, keep, bytes;
};

__host__ __device__ inline DpLds dp_lds(int nops, int ncell, int arena, int cand)
{
    DpLds l;
    int o = 0;
    auto take = [&](int bytes) {
        const int at = o;
        o += (bytes + 7) / 8 * 8;
        return at;
    };
    l.ops = take(32 * nops);
    l.arT = take(8 * arena);
    l.arE = take(8 * arena);
    l.cT = take(8 * cand);
    l.cE = take(8 * cand);
    l.sT = take(8 * kSlots);
    l.sE = take(8 * kSlots);
    l.soff = take(4 * (kSlots + 1));
    l.sstart = take(4 * kSlots);
    l.arB = take(2 * arena);
    l.cstart = take(2 * ncell);
    l.ccnt = take(2 * ncell);
    l.csrc = take(cand);
    l.keep = take(cand);
    l.bytes = o;
    return l;
}

// One instance by one wave, with an arena of `arena` points and `cand` candidates per
// cell; false (nothing written) if the instance needs more.
__device__ bool dp_solve(const DpArgs &a, int64_t inst, char *lds, int arena, int cand)
{
    const int lane = threadIdx.x;
    const int nops = a.I + a.J, W = a.J + 1;
    const DpLds L = dp_lds(nops, (a.I + 1) * W, arena, cand);
    double *ops = (double *)(lds + L.ops);
    double *arT = (double *)(lds + L.arT), *arE = (double *)(lds + L.arE);
    double *cT = (double *)(lds + L.cT), *cE = (double *)(lds + L.cE);
    double *sT = (double *)(lds + L.sT), *sE = (double *)(lds + L.sE);
    int32_t *soff = (int32_t *)(lds + L.soff), *sstart = (int32_t *)(lds + L.sstart);
    int16_t *arB = (int16_t *)(lds + L.arB);
    int16_t *cstart = (int16_t *)(lds + L.cstart), *ccnt = (int16_t *)(lds + L.ccnt);
    uint8_t *keep = (uint8_t *)(lds + L.keep);
    uint8_t *csrc = (uint8_t *)(lds + L.csrc);  // source of each candidate of the cell
    for (int x = lane; x < 4 * nops; x += 64) ops[x] = a.ops[inst * 4 * nops + x];
    if (lane == 0) {
        const int last = a.I * W + a.J;
        arT[0] = 0.0;
        arE[0] = 0.0;
        arB[0] = -1;
        cstart[last] = 0;
        ccnt[last] = 1;
    }
    wave_sync();
    int used = 1;  // arena points in use (uniform)
    bool ok = true;
    for (int i = a.I; i >= 0 && ok; --i) {
        for (int j = a.J; j >= 0 && ok; --j) {
            if (i == a.I && j == a.J) continue;
            const Slots s = dp_slots(a, i, j);
            // lane = decision slot in canonical order; allowed slots become sources
            bool allowed = false;
            double gT = 0.0, gE = 0.0;
            int ni = 0, nj = 0;
            if (lane == 0 && s.va) {
                allowed = true;
                dp_alone(ops + 4 * i, a.p_static, &gT, &gE);
                ni = i + 1;
                nj = j;
            } else if (lane == 1 && s.vb) {
                allowed = true;
                dp_alone(ops + 4 * (a.I + j), a.p_static, &gT, &gE);
                ni = i;
                nj = j + 1;
            } else if (lane >= 2 && lane < 2 + KR_DP_MAX_K && lane - 1 <= s.nc) {
                const int k = lane - 1;
                allowed = true;
                dp_group(ops, i, a.I + j, k, a.p_static, &gT, &gE);
                ni = i + 1;
                nj = j + k;
            } else if (lane >= 2 + KR_DP_MAX_K && lane < kSlots &&
                       lane - 1 - KR_DP_MAX_K <= s.nd) {
                const int k = lane - 1 - KR_DP_MAX_K;
                allowed = true;
                dp_group(ops, a.I + j, i, k, a.p_static, &gT, &gE);
                ni = i + k;
                nj = j + 1;
            }
            const uint64_t m = __ballot(allowed);
            const int ns = __popcll(m);
            const int r = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
            const int n_succ = allowed ? ccnt[ni * W + nj] : 0;
            // exclusive prefix of the successor counts in source order
            int inc = n_succ;
            for (int d = 1; d < 64; d <<= 1) {
                const int y = __shfl_up(inc, d, 64);
                if (lane >= d) inc += y;
            }
            const int C = __shfl(inc, 63, 64);
            if (C > cand) {
                ok = false;
                break;
            }
            const int ex = inc - n_succ;  // first candidate of this lane's source
            const int st = allowed ? (int)cstart[ni * W + nj] : 0;
            int kept;
            if (C <= 64) {
                // one candidate per lane; its source found and read through lane reads
                const bool live = lane < C;
                int sl = 0, sr = 0, rk = 0;
                for (uint64_t mm = m; mm; mm &= mm - 1) {
                    const int l = __ffsll((long long)mm) - 1;
                    if (__builtin_amdgcn_readlane(ex, l) <= lane) {
                        sl = l;
                        sr = rk;
                    }
                    ++rk;
                }
                const double sgT = bitsd(shfl_u64(dbits(gT), sl));
                const double sgE = bitsd(shfl_u64(dbits(gE), sl));
                const int q = lane - __shfl(ex, sl, 64);
                const int sst = __shfl(st, sl, 64);
                double t = INFINITY, e = INFINITY;
                const int lo = sr;
                if (live) {
                    t = sgT + arT[sst + q];
                    e = sgE + arE[sst + q];
                }
                bool k = live;
                for (int y = 0; y < C; ++y) {
                    const double ty = bitsd(lane_u64(dbits(t), y));
                    const double ey = bitsd(lane_u64(dbits(e), y));
                    const bool before = ty < t || (ty == t && (ey < e || (ey == e && y < lane)));
                    if (before && ey <= e) k = false;
                }
                uint64_t km = __ballot(k);
                kept = __popcll(km);
                if (kept > KR_DP_CELL_CAP || used + kept > arena) {
                    ok = false;
                    break;
                }
                int rank = 0;  // kept points are strictly ordered in time
                while (km) {
                    const int y = __ffsll((long long)km) - 1;
                    km &= km - 1;
                    rank += bitsd(lane_u64(dbits(t), y)) < t ? 1 : 0;
                }
                if (k) {
                    arT[used + rank] = t;
                    arE[used + rank] = e;
                    arB[used + rank] = (int16_t)(lo * 64 + q);
                }
            } else {
                if (allowed) {
                    sT[r] = gT;
                    sE[r] = gE;
                    soff[r] = ex;
                    sstart[r] = st;
                    for (int q = 0; q < n_succ; ++q) csrc[ex + q] = (uint8_t)r;
                }
                if (lane == 0) soff[ns] = C;
                wave_sync();
                for (int c = lane; c < C; c += 64) {
                    const int lo = csrc[c];
                    const int q = c - soff[lo];
                    cT[c] = sT[lo] + arT[sstart[lo] + q];
                    cE[c] = sE[lo] + arE[sstart[lo] + q];
                }
                wave_sync();
                int kept_here = 0;
                for (int c = lane; c < C; c += 64) {
                    const double t = cT[c], e = cE[c];
                    bool k = true;
#pragma unroll 4
                    for (int y = 0; y < C; ++y) {
                        const double ty = cT[y], ey = cE[y];
                        const bool before = ty < t || (ty == t && (ey < e || (ey == e && y < c)));
                        if (before && ey <= e) k = false;
                    }
                    keep[c] = k;
                    kept_here += k;
                }
                wave_sync();
                kept = kept_here;
                for (int d = 32; d > 0; d >>= 1) kept += __shfl_xor(kept, d, 64);
                if (kept > KR_DP_CELL_CAP || used + kept > arena) {
                    ok = false;
                    break;
                }
                for (int c = lane; c < C; c += 64) {
                    if (!keep[c]) continue;
                    const double t = cT[c];
                    int rank = 0;
#pragma unroll 4
                    for (int y = 0; y < C; ++y) rank += keep[y] && cT[y] < t;
                    const int lo = csrc[c];
                    arT[used + rank] = t;
                    arE[used + rank] = cE[c];
                    arB[used + rank] = (int16_t)(lo * 64 + (c - soff[lo]));
                }
            }
            if (lane == 0) {
                cstart[i * W + j] = (int16_t)used;
                ccnt[i * W + j] = (int16_t)kept;
            }
            used += kept;
            wave_sync();
        }
    }
    if (!ok) return false;
    const int n0 = ccnt[0];
    if (lane == 0) a.out_n[inst] = n0;
    const int q = lane;
    if (q < n0 && q < a.out_cap) {
        const int64_t o = inst * a.out_cap + q;
        a.out_T[o] = arT[cstart[0] + q];
        a.out_E[o] = arE[cstart[0] + q];
        if (a.out_sched) {
            int32_t *sc = a.out_sched + o * nops;
            int ci = 0, cj = 0, cq = q, d = 0;
            while (!(ci == a.I && cj == a.J) && d < nops) {
                const int b = arB[cstart[ci * W + cj] + cq];
                int ni, nj;
                sc[d++] = dp_decode(a, ci, cj, b / 64, &ni, &nj);
                ci = ni;
                cj = nj;
                cq = b % 64;
            }
            for (; d < nops; ++d) sc[d] = -1;
        }
    }
    return true;
}

__global__ void dp_init_kernel(int32_t *status, int32_t *retry_n)
{
    *status = KR_OK;
    retry_n[0] = 0;
    retry_n[1] = 0;
}

// Every instance with the small on-chip budget; the ones that need more are queued.
__global__ void __launch_bounds__(64) dp_first_kernel(DpArgs a)
{
    extern __shared__ double dp_smem[];
    const int64_t inst = blockIdx.x;
    if (!dp_solve(a, inst, (char *)dp_smem, a.arena_s, a.cand_s) && threadIdx.x == 0) {
        a.out_n[inst] = -1;
        a.retry[atomicAdd(a.retry_n, 1)] = (int32_t)inst;
    }
}

// The instances of queue `tier` (0 or 1) with a larger budget (persistent grid over the
// queue); the ones that still do not fit go to the next queue, or are reported after
// the last tier.
__global__ void __launch_bounds__(64) dp_retry_kernel(DpArgs a, int tier, int arena, int cand)
{
    extern __shared__ double dp_smem[];
    const int n = a.retry_n[tier];
    const int32_t *q = a.retry + (int64_t)tier * a.n_inst;
    for (int r = blockIdx.x; r < n; r += gridDim.x) {
        const int64_t inst = q[r];
        if (!dp_solve(a, inst, (char *)dp_smem, arena, cand) && threadIdx.x == 0) {
            a.out_n[inst] = -1;
            if (tier == 0)
                a.retry[a.n_inst + atomicAdd(a.retry_n + 1, 1)] = (int32_t)inst;
            else
                *a.status = KR_ECAPACITY;
        }
        wave_sync();
    }
}

}  // namespace

hipError_t launch_dp(const DpArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(dp_init_kernel, dim3(1), dim3(1), 0, st, a.status, a.retry_n);
    if (a.n_inst > 0) {
        const int nops = a.I + a.J, ncell = (a.I + 1) * (a.J + 1);
        const int small = dp_lds(nops, ncell, a.arena_s, a.cand_s).bytes;
        hipLaunchKernelGGL(dp_first_kernel, dim3((unsigned)a.n_inst), dim3(64), small, st, a);
        // middle budget: still several instances per compute unit; then the full one
        const int am = KR_DP_ARENA / 2, cm = KR_DP_CAND / 4;
        const int mid = dp_lds(nops, ncell, am, cm).bytes;
        const int big = dp_lds(nops, ncell, KR_DP_ARENA, KR_DP_CAND).bytes;
        const int64_t g1 = a.n_inst < 2048 ? a.n_inst : 2048;
        const int64_t g2 = a.n_inst < 512 ? a.n_inst : 512;
        hipLaunchKernelGGL(dp_retry_kernel, dim3((unsigned)g1), dim3(64), mid, st, a, 0, am, cm);
        hipLaunchKernelGGL(dp_retry_kernel, dim3((unsigned)g2), dim3(64), big, st, a, 1,
                           KR_DP_ARENA, KR_DP_CAND);
    }
    return hipGetLastError();
}

}  // namespace kr
