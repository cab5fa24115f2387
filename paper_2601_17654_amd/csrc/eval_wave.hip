// One-comm candidate evaluation and frontier filter, one wavefront per slab (gfx950).
//
// With one comm kernel the candidates of a (partition, frequency) slab are the launch
// positions x SM choices (Section 4.1).  A 64-lane wave owns a slab at a time: lane
// (h, s) takes SM choice s and the h-th run of consecutive launch positions.  The
// slab's time and power tables are copied from HBM straight into LDS (global_load_lds,
// no register round trip); the copy of the next slab is issued as soon as the current
// one has been evaluated, so it is in flight while the wave filters.  A block is one
// wave, so nothing waits on a barrier.
//
// Running sums (prefix sums of time and energy along the kernel order, one column per
// SM state) are carried by two cursors per lane instead of a table: the launch cursor
// holds A[p], B[p] of the lane's comm-time SM state, the end cursor A[j], B[j] where j
// is the kernel during which the comm kernel ends.  A later launch never ends in an
// earlier kernel, so both cursors only move forward and every sum is formed by the
// same left-to-right additions as the running-sum definition.  The all-SM column's
// sums are formed once per slab and kept in LDS.  The cost arithmetic is the walk of
// the partition cost model (fluid SM-share reading of Sections 3.2 and 4.2) for one
// comm kernel, each line one IEEE fp64 rounding in a fixed order (no FMA contraction).
//
// Frontier of a chunk of the slab (GetFrontier, Algorithm 1): A = least candidate in
// (T, E, index) order, Z = least in (E, T, index) order.  Every kept point other than
// A and Z lies strictly inside their box (T < T_Z, E < E_A), which holds few
// candidates; those are taken by repeated lexicographic minima below the last kept
// energy.  All of it runs on registers with wave reductions.
#include "kr_filter.h"
#include "kr_launch.h"
#include "kr_wave.h"

namespace kr {

typedef __attribute__((address_space(3))) void lds_void;

// Compiler-level ordering of LDS accesses within the wave (the hardware executes one
// wave's LDS instructions in order).
__device__ __forceinline__ void wave_lds_fence()
{
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
}

// Keeps the compiler from sinking the computation of x past this point (it would keep
// the inputs of every unrolled round alive at once).
__device__ __forceinline__ void pin(double &x) { asm volatile("" : "+v"(x)); }

// s_waitcnt encodings (gfx9): vmcnt [3:0]+[15:14], expcnt [6:4], lgkmcnt [11:8].
#define KR_WAIT_VM0 0x0F70
#define KR_WAIT_LGKM0 0xC07F

// Copy n doubles from global memory into LDS, W bytes per lane and instruction (W = 16
// needs n even and both addresses 16-byte aligned).  Lane i of an instruction writes
// LDS bytes [base + W*i, base + W*(i+1)).
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
    if (threadIdx.x == 0) {
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
    const int lane = threadIdx.x;
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

// What a round leaves for its tail, which runs one round later so that the loads it
// needs are in flight meanwhile.
struct Tail {
    int j;
    bool valid;
    double ec;        // B0[p] + (B[j] - B[p])
    double rem;       // comm time left when compute reaches kernel j
    double tau;       // A0[p] + comm time
    double tj, wj;    // t[j][sg], pw[j][sg]
    double t0, w0;    // t[j][0], pw[j][0]
    ColRec cj, c1;    // records j and j + 1
};

// Rest of the walk after the comm kernel (compute back in the all-SM state), written
// without branches.  When the comm kernel outlasts compute (j == N) the same lines
// give T = tau and E_c = ec exactly: row N is a pad row (t = +inf, pw = 0), so w = 1,
// nothing is added but +0, and record N holds the totals.  Invalid rounds give +inf.
__device__ __forceinline__ void finish_tail(const Tail &q, double p_static, double ctail,
                                            double a0, double b0, double &T_out, double &E_out)
{
    double Ec = q.ec + q.wj * q.rem;
    const double w = __builtin_fmax(1.0 - q.rem / q.tj, 0.0);
    const bool part = w < 1.0;  // kernel j is left partly done: finish it in state 0
    const double need = w * q.t0;
    const double used = part ? need : 0.0;
    Ec = Ec + q.w0 * used;
    const double Ai = part ? q.c1.a : q.cj.a, Bi = part ? q.c1.b : q.cj.b;
    Ec = Ec + (b0 - Bi);
    const double el = used + (a0 - Ai);
    const double T = q.tau + el;
    double E = p_static * T;
    E = E + Ec;
    E = E + ctail;
    T_out = q.valid ? T : INFINITY;
    E_out = q.valid ? E : INFINITY;
}

// Block (p, b): one wave, partition p, frequencies [b*fb, min(F, (b+1)*fb)).  LDS:
// t slab [N + KR_PAD][S1] at 0, pw slab (same shape) at w_pw, all-SM column sums
// [N + 2] at w_a0.  The pad rows hold t = +inf (pw = 0), so an end-cursor search that
// runs past the last kernel stops by itself.  SC > 0 fixes the number of SM choices at
// compile time (row offsets become immediates).
//
// Lane (h, s) takes positions [plo, phi): runs of `span` positions (a multiple of 8
// when there are several runs), the last run taking the rest.  Round r of a chunk
// evaluates position c0 + r of every lane.  Its end-cursor search reads a batch of K
// rows loaded one round earlier; the loads for its tail and for the next round are
// issued right after the search, and the previous round's tail is finished while they
// are in flight.  Cursors of a lane past its last position keep moving (their results
// are discarded); only their LDS addresses are clamped.
template <int R, int W, int SC>
__global__ void __launch_bounds__(64) eval_filter_wave_kernel(EvalArgs a, UnitOut o)
{
    constexpr int K = KR_PAD;
    extern __shared__ double lds[];
    const int N = a.N, S = SC > 0 ? SC : a.S, S1 = S + 1, slab = N * S1;
    double *Lt = lds, *Lp = lds + a.w_pw;
    ColRec *C0 = (ColRec *)(lds + a.w_a0);
    const int lane = threadIdx.x;
    const int p = blockIdx.x / a.nfb, fbk = blockIdx.x - p * a.nfb;
    const int f0 = fbk * a.fb, f1 = min(a.F, f0 + a.fb);
    const int s = lane % S, h = lane / S, sg = s + 1;
    const bool on = h < a.H;
    const int plo = on ? min(a.n_pos, h * a.span) : 0;
    const int phi = on ? (h == a.H - 1 ? a.n_pos : min(a.n_pos, plo + a.span)) : 0;
    const size_t slot0 = (size_t)p * a.C + (size_t)f0 * a.Cf;
    double *oT = o.T + slot0, *oE = o.E + slot0;
    int32_t *oI = o.I + slot0;
    int count = 0;
    const double *Ct = Lt + sg;  // column sg of the time table; pw at + w_pw
    const int pwo = a.w_pw;
    // filter scratch, all in the pad rows (restored after use): T in the time pad, E
    // in the power pad, indices after E in the power pad (a power pad of zeros reads
    // back the same whether as doubles or as pairs of zero ints).  The column sums
    // are not touched: a run of several chunks reads them again after a filter.
    const Scratch sc{Lt + slab, Lp + slab, (int32_t *)(Lp + slab + a.wcap), a.wcap};

    // pad rows and the zero record (never overwritten by the slab copies)
    for (int x = lane; x < K * S1; x += 64) {
        Lt[slab + x] = INFINITY;
        Lp[slab + x] = 0.0;
    }
    if (lane == 0) C0[N + 1] = ColRec{0.0, 0.0};

    {
        const size_t pf = (size_t)p * a.F + f0;
        copy_to_lds<W>(a.t + pf * slab, Lt, slab);
        copy_to_lds<W>(a.pw + pf * slab, Lp, slab);
    }
    double tc_next = a.tc[((size_t)p * a.F + f0) * S + s];
    double pc_next = a.pc[((size_t)p * a.F + f0) * S + s];
    for (int f = f0; f < f1; ++f) {
        __builtin_amdgcn_s_waitcnt(KR_WAIT_VM0);  // slab f is in LDS
        wave_lds_fence();
        const double tcm = tc_next;
        const double ctail = pc_next * tc_next;

        // Running sums, 8 rows at a time: every lane sums its column (lane 0 the all-SM
        // column, writing the records; the others their comm-time column) and keeps the
        // sums at its first position, which is a multiple of 8 (or 0).
        double pA = 0.0, pB = 0.0, a0, b0;
        {
            const int cc = lane == 0 ? 0 : sg;
            double sa = 0.0, sb = 0.0;
            for (int i0 = 0; i0 < N; i0 += 8) {
                const double *bt = Lt + (i0 * S1 + cc), *bw = Lp + (i0 * S1 + cc);
                double vt[8], vw[8], ra[8], rb[8];
                if (i0 + 8 <= N) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        vt[q] = bt[q * S1];
                        vw[q] = bw[q * S1];
                    }
                } else {
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        vt[q] = i0 + q < N ? bt[q * S1] : 0.0;
                        vw[q] = i0 + q < N ? bw[q * S1] : 0.0;
                    }
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    ra[q] = sa;
                    rb[q] = sb;
                    sa = sa + vt[q];  // rows past N add +0: exact
                    sb = sb + vw[q] * vt[q];
                }
                if (i0 + 8 == plo) {
                    pA = sa;
                    pB = sb;
                }
                if (lane == 0) {
                    double *c = (double *)(C0 + i0);
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        if (i0 + q < N) {
                            c[2 * q] = ra[q];
                            c[2 * q + 1] = rb[q];
                        }
                }
            }
            if (lane == 0) {
                ((double *)(C0 + N))[0] = sa;
                ((double *)(C0 + N))[1] = sb;
            }
            a0 = bitsd(lane_u64(dbits(sa), 0));
            b0 = bitsd(lane_u64(dbits(sb), 0));
        }
        wave_lds_fence();

        int j = plo;  // end cursor
        double jA = pA, jB = pB;
        for (int ch = 0; ch < a.nch; ++ch) {
            const int c0 = plo + ch * R;
            const int nv = max(0, min(R, phi - c0));
            double vT[R], vE[R];
            double bt[K], bw[K], qt, qw, sA, sB;  // inputs of the next round
            auto load_batch = [&](int jb) {  // rows jb .. jb + K - 1 of column sg
                const double *b0p = Ct + __umul24(jb, S1);
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    bt[k] = b0p[k * S1];
                    bw[k] = b0p[k * S1 + pwo];
                }
            };
            load_batch(min(max(j, c0), N));
            {
                const int pr = max(c0 - 1, 0);
                qt = Ct[__umul24(pr, S1)];
                qw = Ct[__umul24(pr, S1) + pwo];
                const ColRec cs = C0[min(c0, N + 1)];
                sA = cs.a;
                sB = cs.b;
            }
            Tail prev;
            double tl = INFINITY, el = INFINITY;  // this lane's least T and E
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int pp = c0 + r;
                const bool valid = r < nv;
                if (r > 0 || ch > 0) {  // launch cursor: A[pp], B[pp] of column sg
                    pA = pA + qt;
                    pB = pB + qw * qt;
                }
                if (j < pp) {
                    j = pp;
                    jA = pA;
                    jB = pB;
                }
                // end cursor: the largest j with A[j] - A[pp] <= tcm
                bool go = valid;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    if (go) {
                        const double nA = jA + bt[k];  // +inf past the last kernel
                        if (nA - pA <= tcm) {
                            jA = nA;
                            jB = jB + bw[k] * bt[k];
                            ++j;
                        } else {
                            go = false;
                        }
                    }
                }
                if (__ballot(go && j < N)) {  // K or more kernels: one row at a time
                    while (go && j < N) {
                        const double t1 = Ct[__umul24(j, S1)], w1 = Ct[__umul24(j, S1) + pwo];
                        const double nA = jA + t1;
                        if (nA - pA <= tcm) {
                            jA = nA;
                            jB = jB + w1 * t1;
                            ++j;
                        } else {
                            go = false;
                        }
                    }
                }
                const int jc = min(j, N);  // j can pass N only on a lane past its positions
                Tail cur;
                cur.j = jc;
                cur.valid = valid;
                cur.ec = sB + (jB - pB);
                cur.rem = tcm - (jA - pA);
                cur.tau = sA + tcm;
                {
                    const int row = __umul24(jc, S1);
                    cur.tj = Ct[row];  // a pad row when j == N
                    cur.wj = Ct[row + pwo];
                    cur.t0 = Lt[row];
                    cur.w0 = Lp[row];
                    cur.cj = C0[jc];
                    cur.c1 = C0[jc + 1];
                }
                if (r + 1 < R) {
                    load_batch(min(max(j, pp + 1), N));
                    const int pr = min(pp, N);
                    qt = Ct[__umul24(pr, S1)];
                    qw = Ct[__umul24(pr, S1) + pwo];
                    const ColRec cs = C0[min(pp + 1, N + 1)];
                    sA = cs.a;
                    sB = cs.b;
                }
                if (r > 0) {
                    finish_tail(prev, a.p_static, ctail, a0, b0, vT[r - 1], vE[r - 1]);
                    tl = vmin(tl, vT[r - 1]);
                    el = vmin(el, vE[r - 1]);
                    pin(vT[r - 1]);
                    pin(vE[r - 1]);
                }
                prev = cur;
            }
            finish_tail(prev, a.p_static, ctail, a0, b0, vT[R - 1], vE[R - 1]);
            tl = vmin(tl, vT[R - 1]);
            el = vmin(el, vE[R - 1]);
            if (ch == a.nch - 1 && f + 1 < f1) {
                // every LDS read of this slab has returned: the next slab may land
                wave_lds_fence();
                __builtin_amdgcn_s_waitcnt(KR_WAIT_LGKM0);
                const size_t pn = (size_t)p * a.F + f + 1;
                copy_to_lds<W>(a.t + pn * slab, Lt, slab);
                copy_to_lds<W>(a.pw + pn * slab, Lp, slab);
                tc_next = a.tc[pn * S + s];
                pc_next = a.pc[pn * S + s];
            }
            const int ibase = f * a.Cf + c0 * S + s;
            count += wave_frontier<R>(vT, vE, tl, el, ibase, S, sc, oT + count, oE + count,
                                      oI + count);
        }
    }
    if (lane == 0) o.cnt[blockIdx.x] = count;
}

template <int R, int SC>
static void launch_wave_r(const EvalArgs &a, const UnitOut &o, size_t lds, hipStream_t st)
{
    const dim3 grid(a.P * a.nfb), block(64);
    if (a.dma16)
        hipLaunchKernelGGL((eval_filter_wave_kernel<R, 16, SC>), grid, block, lds, st, a, o);
    else
        hipLaunchKernelGGL((eval_filter_wave_kernel<R, 4, SC>), grid, block, lds, st, a, o);
}

hipError_t launch_eval_filter_wave(const EvalArgs &a, const UnitOut &o, hipStream_t st)
{
    const size_t lds = (size_t)a.lds_doubles * sizeof(double);
    if (a.S == 32 && a.R == 17) launch_wave_r<17, 32>(a, o, lds, st);
    else if (a.S == 16 && a.R == 8) launch_wave_r<8, 16>(a, o, lds, st);
    else if (a.S == 8 && a.R == 8) launch_wave_r<8, 8>(a, o, lds, st);
    else {
        switch (a.R) {
        case 2: launch_wave_r<2, 0>(a, o, lds, st); break;
        case 4: launch_wave_r<4, 0>(a, o, lds, st); break;
        case 8: launch_wave_r<8, 0>(a, o, lds, st); break;
        case 17: launch_wave_r<17, 0>(a, o, lds, st); break;
        default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

}  // namespace kr
