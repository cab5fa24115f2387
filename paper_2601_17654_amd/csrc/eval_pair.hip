// Two-comm candidate evaluation and frontier filter, a few waves per slab (gfx950).
//
// With two comm kernels the candidates of a (partition, frequency) slab are the
// launch-position pairs p1 <= p2 times the SM choices (s1, s2) (Sections 4.1, 4.5).  The
// waves of a block share one slab's tables in LDS and split its launch positions p1;
// lane s1 * S + s2 takes SM choices (s1, s2) (at most 8 SM choices, so S * S <= 64) and
// steps through a wave's pairs in candidate order, one pair per round for every lane.
//
// The walk of the partition cost model (fluid SM-share reading of Sections 3.2, 4.2
// and 4.5; the comm kernels share one stream in launch order) falls into phases whose
// inputs repeat across many candidates:
//  - compute in the all-SM state up to kernel p1, then the first comm phase (state
//    s1 + 1 for tc1 seconds), depend on (p1, s1) only;
//  - if compute has not reached kernel p2 when the first comm kernel ends, it runs in
//    the all-SM state up to p2 and the second comm phase starts there with kernel p2
//    untouched: that phase and the all-SM rest after it depend on (p2, s2) only, and
//    are tabled in LDS once per slab;
//  - otherwise the second comm kernel starts as soon as the first ends and continues
//    the first phase's progress: that phase depends on (p1, s1, s2), and each lane
//    forms it once per p1.
// A phase is kept as the values it adds to the energy sum and to the time, in the
// order the walk adds them.  A candidate applies them to its own sums in that order,
// so every candidate gets the roundings of the plain walk, operation for operation.
// A step the walk skips is stored as +0: the energy and time sums are never -0 (they
// start from +0 or a positive value and only non-negative terms are added), so adding
// +0 leaves them unchanged.
#include "kr_filter.h"
#include "kr_launch.h"
#include "kr_wave.h"

namespace kr {

// What a second comm phase and the all-SM rest after it add: energy terms ea (the
// kernel that was in progress), eb (whole kernels), ec (the kernel the phase ends in),
// a4 (the rest finishing that kernel), b4 (the rest's whole kernels), and the rest's
// time el4.  All +0 where the walk adds nothing (ea of a phase starting at a kernel
// boundary; a4, b4, el4 when compute finishes before the comm kernel does).
struct alignas(16) PairRec {
    double ea, eb, ec, a4, b4, el4;
};

// Largest j in [i0, N] with A[j][s] - base <= rb, where base = A[i0][s] and rb >= 0:
// galloping, then bisection.  The predicate is monotone in j (the running sums never
// decrease and rounding is monotone), so this is the j at which a left-to-right scan
// of whole kernels stops.
__device__ __forceinline__ int pair_scan(const ColRec *AB, int S1, int s, int i0, int N,
                                         double base, double rb)
{
    int lo = i0, step = 1;
    while (lo + step <= N && AB[(lo + step) * S1 + s].a - base <= rb) {
        lo += step;
        step <<= 1;
    }
    int hi = min(N, lo + step - 1);
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (AB[mid * S1 + s].a - base <= rb) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Second comm phase in SM state s for tc seconds, from kernel i with unfinished
// fraction w (w = 1: kernel i not started), then the rest in the all-SM state; i < N.
// The lines are the walk's: finish the interrupted kernel if the budget allows (else
// spend the whole budget on it), whole kernels while they fit, the part of the next one
// the budget leaves; then the rest of the interrupted kernel and the remaining kernels.
__device__ __forceinline__ PairRec pair_phase(const double *Lt, const double *Lp,
                                              const ColRec *AB, int S1, int N, int s, int i,
                                              double w, double tc)
{
    PairRec o{0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    double used = 0.0;
    bool fin = false, spent = false;
    if (w < 1.0) {
        const double tk = Lt[i * S1 + s];
        const double need = w * tk;
        if (need <= tc) {
            o.ea = Lp[i * S1 + s] * need;
            used = need;
            i = i + 1;
            w = 1.0;
        } else {  // the budget ends inside the interrupted kernel
            o.ea = Lp[i * S1 + s] * tc;
            w = w - tc / tk;
            if (w < 0.0) w = 0.0;
            spent = true;
        }
    }
    if (!spent) {
        const double rb = tc - used;
        const ColRec zi = AB[i * S1 + s];
        const int j = pair_scan(AB, S1, s, i, N, zi.a, rb);
        const ColRec zj = AB[j * S1 + s];
        o.eb = zj.b - zi.b;
        if (j == N) {
            fin = true;
        } else {
            const double r = rb - (zj.a - zi.a);
            o.ec = Lp[j * S1 + s] * r;
            w = 1.0 - r / Lt[j * S1 + s];
            if (w < 0.0) w = 0.0;
            i = j;
        }
    }
    if (!fin) {  // the rest in the all-SM state (column 0)
        double u = 0.0;
        if (w < 1.0) {
            const double need = w * Lt[i * S1];
            o.a4 = Lp[i * S1] * need;
            u = need;
            i = i + 1;
        }
        const ColRec zN = AB[N * S1], zi = AB[i * S1];
        o.b4 = zN.b - zi.b;
        o.el4 = u + (zN.a - zi.a);
    }
    return o;
}

// Sorts n keys (T bits, E bits, index) ascending in LDS by one wave: a bitonic network
// whose comparators all put the smaller key at the lower index (the first stage of each
// merge compares mirrored positions); entries from n on act as +inf and never move.
__device__ inline void wave_sort_keys(uint64_t *sT, uint64_t *sE, int32_t *sI, int n)
{
    int m = 1, lm = 0;
    while (m < n) {
        m <<= 1;
        ++lm;
    }
    for (int lk = 1; lk <= lm; ++lk) {
        const int k = 1 << lk;
        for (int lj = lk - 1; lj >= 0; --lj) {
            const int j = 1 << lj;
            for (int q = threadIdx.x & 63; q < (m >> 1); q += 64) {
                int lo, hi;
                if (lj == lk - 1) {
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
                        sT[lo] = tb;
                        sE[lo] = eb;
                        sI[lo] = ib;
                        sT[hi] = ta;
                        sE[hi] = ea;
                        sI[hi] = ia;
                    }
                }
            }
            wave_lds_fence();
        }
    }
}

// GetFrontier's strict prefix minimum over n keys sorted by (T, E, index), by one wave:
// writes the keys whose E is below every earlier E to o*[0 ..) in order and returns
// their count (uniform).  Lane l scans a contiguous block of the keys.
__device__ inline int wave_frontier_scan(const uint64_t *sT, const uint64_t *sE, const int32_t *sI,
                                         int n, double *oT, double *oE, int32_t *oI)
{
    const int lane = threadIdx.x & 63;
    const int per = (n + 63) / 64;
    const int q0 = min(n, lane * per), q1 = min(n, q0 + per);
    uint64_t m = KR_INF_BITS;
    for (int q = q0; q < q1; ++q) m = min(m, sE[q]);
    unsigned long long inc = m;  // least E of lanes 0 .. lane
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const unsigned long long y = __shfl_up(inc, d, 64);
        if (lane >= d) inc = min(inc, y);
    }
    unsigned long long best0 = __shfl_up(inc, 1, 64);  // least E of the lanes before
    if (lane == 0) best0 = KR_INF_BITS;
    uint64_t best = best0;
    int nk = 0;
    for (int q = q0; q < q1; ++q)
        if (sE[q] < best) {
            ++nk;
            best = sE[q];
        }
    int pos = nk;  // kept keys of lanes 0 .. lane
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(pos, d, 64);
        if (lane >= d) pos += y;
    }
    const int total = __builtin_amdgcn_readlane(pos, 63);
    pos -= nk;
    best = best0;
    for (int q = q0; q < q1; ++q) {
        const uint64_t e = sE[q];
        if (e < best) {
            oT[pos] = bitsd(sT[q]);
            oE[pos] = bitsd(e);
            oI[pos] = sI[q];
            ++pos;
            best = e;
        }
    }
    return total;
}

// The wave of a block of NW waves that takes launch position p1 (snake order).
__host__ __device__ __forceinline__ int pair_owner(int p1, int NW)
{
    const int r = p1 % (2 * NW);
    return r < NW ? r : 2 * NW - 1 - r;
}

// Copy n doubles from global memory into LDS by the block's NW waves, W bytes per lane
// and instruction (W = 16 needs n even and both addresses 16-byte aligned).
template <int W, int NW>
__device__ __forceinline__ void copy_to_lds_nw(const double *g, double *l, int n)
{
    const int units = n * 8 / W;
    const int lane = threadIdx.x & 63, w0 = threadIdx.x & ~63;
    for (int u0 = w0; u0 < units; u0 += 64 * NW) {
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

// Block (p, b): NW waves sharing the slabs of partition p, frequencies [b*fb,
// min(F, (b+1)*fb)), one slab at a time.  LDS (in doubles): t slab [N][S1] at 0, pw slab
// at q_pw, running sums {A, B} [N + 1][S1] at q_ab (column 0 the all-SM state), the
// fresh second-phase table [n_pos][S] at q_f, each wave's continuing second phases [64]
// at q_c, each wave's filter scratch at q_sc.  Launch positions p1 go to the waves in
// snake order (0, 1, .., NW - 1, NW - 1, .., 0, 0, 1, ..), which evens out the pairs
// each wave takes; a wave is a unit of its own (slot and count), so waves never share
// output.
// Round r of a chunk evaluates pair (p1, c0 + r) for every lane; pairs past the last
// position are clamped for the loads and give +inf.  Each chunk's frontier goes to the
// wave's slot; at the end of a slab those points (usually many times the slab's own
// frontier) are read back into the second-phase tables, idle by then, sorted, and
// replaced in place by their frontier, when they fit there.  SC > 0 fixes the number of
// SM choices at compile time; FN also fixes the two-comm workload's 48 kernels and 33
// launch positions.
template <int R, int W, int NW, int SC, bool FN>
__global__ void __launch_bounds__(64 * NW) eval_filter_pair_kernel(EvalArgs a, UnitOut o)
{
    extern __shared__ __attribute__((aligned(16))) double lds[];
    static_assert(!FN || SC > 0, "the fixed shape fixes the SM choices too");
    const int N = FN ? 48 : a.N, S = SC > 0 ? SC : a.S, S1 = S + 1, SS = S * S, slab = N * S1;
    const int np = FN ? 33 : a.n_pos;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double *const Lt = lds, *const Lp = lds + a.q_pw;
    ColRec *const AB = (ColRec *)(lds + a.q_ab);
    PairRec *const Fr = (PairRec *)(lds + a.q_f);
    PairRec *const Cw = (PairRec *)(lds + a.q_c) + 64 * wave;
    double *const scw = lds + a.q_sc + 160 * wave;
    const Scratch sc{scw, scw + 64, (int32_t *)(scw + 128), 64};
    const int p = blockIdx.x / a.nfb, fbk = blockIdx.x - p * a.nfb;
    const int f0 = fbk * a.fb, f1 = min(a.F, f0 + a.fb);
    const bool live = lane < SS;
    const int s1 = live ? lane / S : 0, s2 = live ? lane - (lane / S) * S : 0;
    // rows of the fresh table this thread forms: SM choice sF, positions g, g + G, ...
    const int G = 64 * NW / S, g = tid / S, sF = tid - g * S;
    const int64_t unit = (int64_t)blockIdx.x * NW + wave;
    const size_t slot0 = (size_t)p * a.useg + (size_t)(unit - (int64_t)p * a.uper) * a.ustride;
    double *const oT = o.T + slot0, *const oE = o.E + slot0;
    int32_t *const oI = o.I + slot0;
    int count = 0;
    const double p_static = a.p_static;
    // sort room of the slab-end reduction: this wave's share of the fresh and continuing
    // tables
    const int scap = a.pair_scap;
    uint64_t *const sT = (uint64_t *)(lds + a.q_f) + (size_t)wave * ((a.q_sc - a.q_f) / NW);
    uint64_t *const sE = sT + scap;
    int32_t *const sI = (int32_t *)(sE + scap);

    for (int f = f0; f < f1; ++f) {
        const size_t pf = (size_t)p * a.F + f;
        const int cs = count;  // first output of this slab
        // every LDS read of the previous slab has returned (all waves: the barrier
        // after the reduction, or none yet)
        copy_to_lds_nw<W, NW>(a.t + pf * slab, Lt, slab);
        copy_to_lds_nw<W, NW>(a.pw + pf * slab, Lp, slab);
        const double *const cm = a.tc + pf * 2 * S, *const cpw = a.pc + pf * 2 * S;
        const double tc1 = cm[s1], tc2 = cm[S + s2], tcF = cm[S + sF];
        const double ct1 = cpw[s1] * tc1, ct2 = cpw[S + s2] * tc2;
        __builtin_amdgcn_s_waitcnt(KR_WAIT_VM0);  // this wave's part of slab f is in LDS
        __syncthreads();                          // and the other waves' parts

        // Running sums, thread c < S1 forming column c left to right (8 rows of loads
        // ahead of the additions).
        if (tid < S1) {
            double sa = 0.0, sb = 0.0;
            AB[tid] = ColRec{0.0, 0.0};
            for (int i0 = 0; i0 < N; i0 += 8) {
                double vt[8], vw[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const int i = min(i0 + q, N - 1);
                    vt[q] = Lt[i * S1 + tid];
                    vw[q] = Lp[i * S1 + tid];
                }
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    if (i0 + q < N) {
                        sa = sa + vt[q];
                        sb = sb + vw[q] * vt[q];
                        AB[(i0 + q + 1) * S1 + tid] = ColRec{sa, sb};
                    }
            }
        }
        __syncthreads();
        // Second comm phases that start fresh at kernel q.  Row q = N (a comm kernel
        // launched after the last compute kernel) adds nothing: all +0.
        if (g < G)
            for (int q = g; q < np; q += G)
                Fr[q * S + sF] = q < N ? pair_phase(Lt, Lp, AB, S1, N, sF + 1, q, 1.0, tcF)
                                       : PairRec{0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
        __syncthreads();

        for (int p1 = 0; p1 < np; ++p1) {
            if (pair_owner(p1, NW) != wave) continue;
            // compute up to p1 in the all-SM state, then the first comm phase
            const int sa1 = s1 + 1;
            const ColRec z0 = AB[p1 * S1], zp = AB[p1 * S1 + sa1];
            const int j1 = p1 < N ? pair_scan(AB, S1, sa1, p1, N, zp.a, tc1) : N;
            const ColRec zj = AB[j1 * S1 + sa1];
            double Ec1 = z0.b + (zj.b - zp.b);
            const double tau1 = z0.a + tc1;
            double w1 = 1.0;
            if (j1 < N) {
                const double r1 = tc1 - (zj.a - zp.a);
                Ec1 = Ec1 + Lp[j1 * S1 + sa1] * r1;
                w1 = 1.0 - r1 / Lt[j1 * S1 + sa1];
                if (w1 < 0.0) w1 = 0.0;
            }
            // compute on to p2 in the all-SM state (candidates with j1 < p2)
            double Eca = Ec1, used2 = 0.0;
            int i2 = j1;
            if (j1 < N && w1 < 1.0) {
                const double need = w1 * Lt[j1 * S1];
                Eca = Ec1 + Lp[j1 * S1] * need;
                used2 = need;
                i2 = j1 + 1;
            }
            const ColRec zi2 = AB[i2 * S1];
            // the second comm phase continuing the first one's progress (p2 <= j1)
            Cw[lane] = j1 < N ? pair_phase(Lt, Lp, AB, S1, N, s2 + 1, j1, w1, tc2)
                              : PairRec{0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
            wave_lds_fence();
            const int ppb = p1 * np - p1 * (p1 - 1) / 2 - p1;  // pair rank of (p1, p2): ppb + p2
            for (int c0 = p1; c0 < np; c0 += R) {
                double vT[R], vE[R];
                double tl = INFINITY, el = INFINITY;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int p2 = min(c0 + r, np - 1);
                    const bool valid = live && c0 + r < np;
                    const bool fresh = j1 < p2;
                    const ColRec z2 = AB[p2 * S1];
                    const PairRec q = *(fresh ? Fr + p2 * S + s2 : Cw + lane);
                    const double EcF = Eca + (z2.b - zi2.b);
                    const double stF = tau1 + (used2 + (z2.a - zi2.a));
                    double Ec = fresh ? EcF : Ec1;
                    const double st2 = fresh ? stF : tau1;
                    Ec = Ec + q.ea;
                    Ec = Ec + q.eb;
                    Ec = Ec + q.ec;
                    Ec = Ec + q.a4;
                    Ec = Ec + q.b4;
                    const double T = (st2 + tc2) + q.el4;
                    double E = p_static * T;
                    E = E + Ec;
                    E = E + ct1;
                    E = E + ct2;
                    vT[r] = valid ? T : INFINITY;
                    vE[r] = valid ? E : INFINITY;
                    tl = vmin(tl, vT[r]);
                    el = vmin(el, vE[r]);
                }
                const int ibase = f * a.Cf + (ppb + c0) * SS + lane;
                count += wave_frontier<R>(vT, vE, tl, el, ibase, SS, sc, oT + count, oE + count,
                                          oI + count);
            }
            wave_lds_fence();  // the continuing phase of this p1 is read
        }
        __syncthreads();  // every wave is done with the slab's tables
        const int ns = count - cs;
        if (ns > 1 && ns <= scap) {
            // this wave's own stores, complete after the wait: plain loads see them
            __builtin_amdgcn_s_waitcnt(KR_WAIT_VM0);
            for (int x = lane; x < ns; x += 64) {
                sT[x] = dbits(oT[cs + x]);
                sE[x] = dbits(oE[cs + x]);
                sI[x] = oI[cs + x];
            }
            wave_lds_fence();
            wave_sort_keys(sT, sE, sI, ns);
            count = cs + wave_frontier_scan(sT, sE, sI, ns, oT + cs, oE + cs, oI + cs);
        }
        __syncthreads();  // the sort room is free again, and Lt, Lp may be overwritten
    }
    if (lane == 0) o.cnt[unit] = count;
}

int pair_owner_host(int p1, int NW) { return pair_owner(p1, NW); }

hipError_t launch_eval_filter_pair(const EvalArgs &a, const UnitOut &o, hipStream_t st)
{
    const size_t lds = (size_t)a.lds_doubles * sizeof(double);
    constexpr int NW = KR_PAIR_WAVES;
    const dim3 grid(a.P * a.nfb), block(64 * NW);
    if (a.dma16 && a.S == 8 && a.N == 48 && a.n_pos == 33)
        hipLaunchKernelGGL((eval_filter_pair_kernel<8, 16, NW, 8, true>), grid, block, lds, st, a, o);
    else if (a.dma16 && a.S == 8)
        hipLaunchKernelGGL((eval_filter_pair_kernel<8, 16, NW, 8, false>), grid, block, lds, st, a, o);
    else if (a.dma16)
        hipLaunchKernelGGL((eval_filter_pair_kernel<8, 16, NW, 0, false>), grid, block, lds, st, a, o);
    else
        hipLaunchKernelGGL((eval_filter_pair_kernel<8, 4, NW, 0, false>), grid, block, lds, st, a, o);
    return hipGetLastError();
}

}  // namespace kr
