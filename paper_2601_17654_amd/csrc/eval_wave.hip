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

__device__ __forceinline__ void emit(const Key &k, int n, double *oT, double *oE, int32_t *oI)
{
    if (threadIdx.x == 0) {
        oT[n] = bitsd(k.t);
        oE[n] = bitsd(k.e);
        oI[n] = k.i;
    }
}

// Frontier of the wave's chunk (invalid slots hold T = E = +inf; valid ones are
// finite).  Candidate index of slot r of a lane is ibase + r * S.  Writes the frontier
// in ascending T to o*[0 .. n) and returns n (uniform).
template <int R>
__device__ inline int wave_frontier(const double (&vT)[R], const double (&vE)[R], int ibase, int S,
                                    double *oT, double *oE, int32_t *oI)
{
    double tl = INFINITY, el = INFINITY;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        tl = vT[r] < tl ? vT[r] : tl;
        el = vE[r] < el ? vE[r] : el;
    }
    const uint64_t TA = wave_min_u64(dbits(tl));
    if (TA == KR_INF_BITS) return 0;
    const uint64_t EZ = wave_min_u64(dbits(el));
    const Key A = chunk_pick<R>(vT, vE, ibase, S, [&](int r) { return dbits(vT[r]) == TA; });
    emit(A, 0, oT, oE, oI);
    if (A.e == EZ) return 1;  // A has the least energy too: nothing beats it
    const Key Z = chunk_pick<R>(vT, vE, ibase, S, [&](int r) { return dbits(vE[r]) == EZ; });
    // candidates strictly inside the box of A and Z
    uint32_t rows = 0;
    int nbox = 0;
    Key one = key_none();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const uint64_t m = __ballot(dbits(vT[r]) < Z.t && dbits(vE[r]) < A.e);
        if (m) {
            rows |= 1u << r;
            nbox += __popcll(m);
            const int L = __ffsll((long long)m) - 1;
            one = Key{lane_u64(dbits(vT[r]), L), lane_u64(dbits(vE[r]), L),
                      lane_i32(ibase, L) + r * S};
        }
    }
    int n = 1;
    if (nbox == 1) {
        emit(one, n++, oT, oE, oI);  // lies below A's energy and before Z: kept
    } else if (nbox > 1) {
        uint64_t bound = A.e;
        for (;;) {
            Key loc = key_none();
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (rows >> r & 1u) {
                    const Key c{dbits(vT[r]), dbits(vE[r]), ibase + r * S};
                    if (c.t < Z.t && c.e < bound && kless(c, loc)) loc = c;
                }
            const Key w = wave_min_key(loc);
            if (w.t == KR_INF_BITS) break;
            emit(w, n++, oT, oE, oI);
            bound = w.e;
        }
    }
    emit(Z, n++, oT, oE, oI);
    return n;
}

// All-SM column record of row i: the running sums before row i and the row's own
// entries.  Record N holds the totals (and zeros).
struct alignas(16) ColRec {
    double a, b;  // A0[i], B0[i]
    double t, w;  // t[i][0], pw[i][0]
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
    ColRec cj;        // record j
    double c1a, c1b;  // sums of record j + 1
};

// Rest of the walk after the comm kernel (compute back in the all-SM state), written
// without branches; results of invalid rounds are +inf.
__device__ __forceinline__ void finish_tail(const Tail &q, int N, double p_static, double ctail,
                                            double a0, double b0, double &T_out, double &E_out)
{
    // comm ends inside kernel j: finish kernel j's remaining fraction, then the rest
    double Ec = q.ec + q.wj * q.rem;
    double w = 1.0 - q.rem / q.tj;
    w = w < 0.0 ? 0.0 : w;
    const bool part = w < 1.0;
    const double need = w * q.cj.t;
    const double Ecp = Ec + q.cj.w * need;
    const double used = part ? need : 0.0;
    Ec = part ? Ecp : Ec;
    const double Ai = part ? q.c1a : q.cj.a, Bi = part ? q.c1b : q.cj.b;
    Ec = Ec + (b0 - Bi);
    const double el = used + (a0 - Ai);
    const double Tin = q.tau + el;
    // j == N: compute finished while the comm kernel ran
    const bool over = q.j == N;
    const double T = over ? q.tau : Tin;
    Ec = over ? q.ec : Ec;
    double E = p_static * T;
    E = E + Ec;
    E = E + ctail;
    T_out = q.valid ? T : INFINITY;
    E_out = q.valid ? E : INFINITY;
}

// Block (p, b): one wave, partition p, frequencies [b*fb, min(F, (b+1)*fb)).  LDS:
// t slab [N + KR_PAD][S1] at 0, pw slab (same shape) at w_pw, all-SM column records
// [N + 2] at w_a0.  The pad rows hold t = +inf (pw = 0), so an end-cursor search that
// runs past the last kernel stops by itself; the last record is zeros.  SC > 0 fixes the
// number of SM choices at compile time (row offsets become immediates).
// Rounds: round r of a chunk evaluates position c0 + r of every lane.  Its end-kernel
// search reads a batch of K rows loaded one round earlier; the loads for its tail and
// for the next round are issued right after the search, and the previous round's tail
// is finished while they are in flight.
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
    const int plo = h < a.H ? min(a.n_pos, h * a.span) : 0;
    const int phi = h < a.H ? min(a.n_pos, plo + a.span) : 0;
    const size_t slot0 = (size_t)p * a.C + (size_t)f0 * a.Cf;
    double *oT = o.T + slot0, *oE = o.E + slot0;
    int32_t *oI = o.I + slot0;
    int count = 0;
    auto col = [&](const double *L, int row) { return L[row * S1 + sg]; };

    // pad rows and the zero record (never overwritten by the slab copies)
    for (int x = lane; x < K * S1; x += 64) {
        Lt[slab + x] = INFINITY;
        Lp[slab + x] = 0.0;
    }
    if (lane == 0) C0[N + 1] = ColRec{0.0, 0.0, 0.0, 0.0};

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

        // Running sums, one instruction stream: lane 0 sums the all-SM column over
        // every row and writes the records; a lane of a later position run sums its own
        // column up to its first position.  Rows are loaded 8 at a time, one block ahead.
        const int ccol = lane == 0 ? 0 : sg;
        const int nrow = lane == 0 ? N : plo;
        double sa = 0.0, sb = 0.0;
        {
            double vt[8], vw[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int i = min(q, N - 1);
                vt[q] = Lt[i * S1 + ccol];
                vw[q] = Lp[i * S1 + ccol];
            }
            for (int i0 = 0; i0 < N; i0 += 8) {
                double nt[8], nw[8];
                if (i0 + 8 < N) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        const int i = min(i0 + 8 + q, N - 1);
                        nt[q] = Lt[i * S1 + ccol];
                        nw[q] = Lp[i * S1 + ccol];
                    }
                }
                double ra[8], rb[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    ra[q] = sa;
                    rb[q] = sb;
                    if (i0 + q < nrow) {
                        sa = sa + vt[q];
                        sb = sb + vw[q] * vt[q];
                    }
                }
                if (lane == 0) {
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        if (i0 + q < N) C0[i0 + q] = ColRec{ra[q], rb[q], vt[q], vw[q]};
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    vt[q] = nt[q];
                    vw[q] = nw[q];
                }
            }
        }
        if (lane == 0) C0[N] = ColRec{sa, sb, 0.0, 0.0};
        const double a0 = bitsd(lane_u64(dbits(sa), 0)), b0 = bitsd(lane_u64(dbits(sb), 0));
        double pA = lane == 0 ? 0.0 : sa, pB = lane == 0 ? 0.0 : sb;
        wave_lds_fence();

        int j = plo;  // end cursor
        double jA = pA, jB = pB;
        double bt[K], bw[K], qt, qw, sA, sB;  // loaded one round ahead
        auto load_next = [&](int pp) {  // inputs of the round at position pp (<= N + 1)
            const double *bt0 = Lt + (min(max(j, pp), N) * S1 + sg);  // rows jb .. jb + K - 1
            const double *bw0 = bt0 + a.w_pw;
#pragma unroll
            for (int k = 0; k < K; ++k) {
                bt[k] = bt0[k * S1];
                bw[k] = bw0[k * S1];
            }
            const int pr = max(pp - 1, 0);  // row of the launch-cursor step
            qt = col(Lt, pr);
            qw = col(Lp, pr);
            const ColRec cs = C0[pp];
            sA = cs.a;
            sB = cs.b;
        };
        load_next(plo);
        for (int ch = 0; ch < a.nch; ++ch) {
            const int c0 = plo + ch * R;
            const int nv = max(0, min(R, phi - c0));
            double vT[R], vE[R];
            Tail prev;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int pp = c0 + r;
                const bool valid = r < nv;
                if (valid && pp > plo) {  // launch cursor: A[pp], B[pp] of column sg
                    pA = pA + qt;
                    pB = pB + qw * qt;
                }
                if (valid && j < pp) {
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
                if (__ballot(go && j < N)) {  // more than K - 1 kernels: one row at a time
                    while (go && j < N) {
                        const double t1 = col(Lt, j), w1 = col(Lp, j);
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
                Tail cur;
                cur.j = j;
                cur.valid = valid;
                cur.ec = sB + (jB - pB);
                cur.rem = tcm - (jA - pA);
                cur.tau = sA + tcm;
                {
                    cur.tj = col(Lt, j);  // a pad row when j == N (unused then)
                    cur.wj = col(Lp, j);
                    cur.cj = C0[j];
                    const ColRec c1 = C0[j + 1];
                    cur.c1a = c1.a;
                    cur.c1b = c1.b;
                }
                if (r + 1 < R || ch + 1 < a.nch) load_next(pp + 1);
                if (r > 0) {
                    finish_tail(prev, N, a.p_static, ctail, a0, b0, vT[r - 1], vE[r - 1]);
                    pin(vT[r - 1]);
                    pin(vE[r - 1]);
                }
                prev = cur;
            }
            finish_tail(prev, N, a.p_static, ctail, a0, b0, vT[R - 1], vE[R - 1]);
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
            count += wave_frontier<R>(vT, vE, ibase, S, oT + count, oE + count, oI + count);
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
    else if (a.S == 8 && a.R == 4) launch_wave_r<4, 8>(a, o, lds, st);
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
