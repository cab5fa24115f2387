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

// Keeps the compiler from sinking the computation of x past this point (it would keep
// the inputs of every unrolled round alive at once).
__device__ __forceinline__ void pin(double &x) { asm volatile("" : "+v"(x)); }

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
// are discarded); only their LDS addresses are clamped.  FX (32 kernels, 33 positions,
// 32 SM choices: runs of 16 and 17 positions) makes the sizes and LDS offsets
// immediates and lets every round but the last skip the validity selects.
template <int R, int W, int SC, bool FX>
__global__ void __launch_bounds__(64) eval_filter_wave_kernel(EvalArgs a, UnitOut o)
{
    constexpr int K = KR_PAD;
    extern __shared__ double lds[];
    static_assert(!FX || (SC == 32 && R == 17), "the fixed layout is the 32 x 32 one");
    const int N = FX ? 32 : a.N, S = SC > 0 ? SC : a.S, S1 = S + 1, slab = N * S1;
    const int nH = FX ? 2 : a.H, nspan = FX ? 16 : a.span;
    const int npos = FX ? 33 : a.n_pos, nch = FX ? 1 : a.nch;
    const int pwo = FX ? KR_FIX32_PW : a.w_pw;  // power table offset (doubles)
    double *Lt = lds, *Lp = lds + pwo;
    ColRec *C0 = (ColRec *)(lds + (FX ? 2 * KR_FIX32_PW : a.w_a0));
    const int lane = threadIdx.x;
    const int p = blockIdx.x / a.nfb, fbk = blockIdx.x - p * a.nfb;
    const int f0 = fbk * a.fb, f1 = min(a.F, f0 + a.fb);
    const int s = lane % S, h = lane / S, sg = s + 1;
    const bool on = h < nH;
    const int plo = on ? min(npos, h * nspan) : 0;
    const int phi = on ? (h == nH - 1 ? npos : min(npos, plo + nspan)) : 0;
    const size_t slot0 = (size_t)p * a.C + (size_t)f0 * a.Cf;
    double *oT = o.T + slot0, *oE = o.E + slot0;
    int32_t *oI = o.I + slot0;
    int count = 0;
    const double *Ct = Lt + sg;  // column sg of the time table; pw at + pwo
    // filter scratch, all in the pad rows (restored after use): T in the time pad, E
    // in the power pad, indices after E in the power pad (a power pad of zeros reads
    // back the same whether as doubles or as pairs of zero ints).  The column sums
    // are not touched: a run of several chunks reads them again after a filter.
    const Scratch sc{Lt + slab, Lp + slab, (int32_t *)(Lp + slab + a.wcap), a.wcap};
    // Row clamps.  With FX every lane's runs end at or before position N and its last
    // round is its only possibly idle one, so the cursors never pass row N and the
    // loads one round ahead never pass row N + 1: the clamps hold by construction.
    auto cap = [&](int x, int hi) { return FX ? x : min(x, hi); };

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
#pragma unroll 1
            for (int i0 = 0; i0 < N; i0 += 8) {
                const double *bt = Lt + (i0 * S1 + cc), *bw = Lp + (i0 * S1 + cc);
                double vt[8], vw[8], ra[8], rb[8];
                if (FX || i0 + 8 <= N) {
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
                        if (FX || i0 + q < N) {
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
        for (int ch = 0; ch < nch; ++ch) {
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
            load_batch(cap(j, N));
            {
                const int pr = max(c0 - 1, 0);
                qt = Ct[__umul24(pr, S1)];
                qw = Ct[__umul24(pr, S1) + pwo];
                const ColRec cs = C0[cap(c0, N + 1)];
                sA = cs.a;
                sB = cs.b;
            }
            Tail prev;
            double tl = INFINITY, el = INFINITY;  // this lane's least T and E
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int pp = c0 + r;
                const bool valid = (FX && r < R - 1) || r < nv;
                if (r > 0 || ch > 0) {  // launch cursor: A[pp], B[pp] of column sg
                    pA = pA + qt;
                    pB = pB + qw * qt;
                }
                // End cursor: the largest j with A[j] - A[pp] <= tcm.  It is at least
                // pp - 1 here; at pp - 1 the first row of the batch moves it to pp, since
                // its sum A[pp] is formed by the same additions as the launch cursor's
                // (the difference is exactly 0, never above the comm time).
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
                // K or more kernels: one row at a time, never past row N (with finite
                // inputs the pad row N stops a cursor by itself; the bound also ends the
                // walk for unchecked inputs such as an infinite comm time)
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
                const int jc = cap(j, N);  // j can pass N only on a lane past its positions
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
                    load_batch(cap(j, N));
                    const int pr = cap(pp, N);
                    qt = Ct[__umul24(pr, S1)];
                    qw = Ct[__umul24(pr, S1) + pwo];
                    const ColRec cs = C0[cap(pp + 1, N + 1)];
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
            if (ch == nch - 1 && f + 1 < f1) {
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

template <int R, int SC, bool FX = false>
static void launch_wave_r(const EvalArgs &a, const UnitOut &o, size_t lds, hipStream_t st)
{
    const dim3 grid(a.P * a.nfb), block(64);
    if (a.dma16)
        hipLaunchKernelGGL((eval_filter_wave_kernel<R, 16, SC, FX>), grid, block, lds, st, a, o);
    else
        hipLaunchKernelGGL((eval_filter_wave_kernel<R, 4, SC, FX>), grid, block, lds, st, a, o);
}

hipError_t launch_eval_filter_wave(const EvalArgs &a, const UnitOut &o, hipStream_t st)
{
    const size_t lds = (size_t)a.lds_doubles * sizeof(double);
    if (a.S == 32 && a.R == 17 && a.fixed32) launch_wave_r<17, 32, true>(a, o, lds, st);
    else if (a.S == 32 && a.R == 17) launch_wave_r<17, 32>(a, o, lds, st);
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
