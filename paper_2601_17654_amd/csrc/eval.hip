// Candidate evaluation on gfx950.
//
// The (kernel x SM-state) slab of the time and power tables for one (partition,
// frequency) is contiguous in HBM.  It is staged into LDS with coalesced loads, the
// per-state running sums of time and energy are formed in LDS (one thread per state
// column, left to right), and the partition cost model is walked for each candidate
// reading only LDS.  In the fused kernel a workgroup owns one partition and a range
// of frequencies: while it evaluates and filters one slab, the next slab is already
// in flight into registers.
//
// Cost model (fluid SM-share reading of Sections 3.2 and 4.2; the paper gives no
// closed form, Section 4.3.1): compute kernels progress at 1/t in the current SM
// state; comm kernel m is launched when compute reaches the start of kernel p_m and
// starts when the comm stream is free (FIFO); while it runs, compute is in state
// s_m + 1.  T = later of compute end and last comm end; E = p_static * T + compute
// dynamic energy + comm dynamic energy (Sections 2.1, 2.3, 4.5).  Every line below
// is one IEEE fp64 rounding in a fixed order; the library is built without FMA
// contraction so the results are reproducible bit for bit.
//
// LDS slab layout (doubles, row-major with row length S1 = S + 1 states):
//   t [N][S1], pw [N][S1], tc [M][S], pc [M][S], A [N+1][S1], B [N+1][S1]
// where A[i][s] = sum_{k<i} t[k][s] and B[i][s] = sum_{k<i} pw[k][s]*t[k][s].
#include "kr_filter.h"
#include "kr_launch.h"

namespace kr {

struct Slab {
    const double *t, *pw, *tc, *pc, *A, *B;
    const int32_t *pairs;  // [n_pp] p1 | p2 << 16 (M = 2)
    int N, S1, S;
};

__device__ __forceinline__ double sA(const Slab &L, int i, int s) { return L.A[i * L.S1 + s]; }
__device__ __forceinline__ double sB(const Slab &L, int i, int s) { return L.B[i * L.S1 + s]; }
__device__ __forceinline__ double sT(const Slab &L, int i, int s) { return L.t[i * L.S1 + s]; }
__device__ __forceinline__ double sP(const Slab &L, int i, int s) { return L.pw[i * L.S1 + s]; }

__device__ __forceinline__ Slab slab_view(const EvalArgs &a, double *lds)
{
    const int S1 = a.S + 1, slab = a.N * S1, ms = a.M * a.S;
    Slab L;
    L.t = lds;
    L.pw = lds + slab;
    L.tc = lds + 2 * slab;
    L.pc = L.tc + ms;
    L.A = L.pc + ms;
    L.B = L.A + (a.N + 1) * S1;
    L.pairs = (const int32_t *)(L.B + (a.N + 1) * S1);
    L.N = a.N;
    L.S1 = S1;
    L.S = a.S;
    return L;
}

// Largest j in [lo, hi] with A[j][s] - base <= rb, given that lo satisfies it (the
// predicate is monotone in j because the running sums never decrease).  Galloping
// from lo, then bisection: the same j as a left-to-right scan.
__device__ __forceinline__ int fit_from(const Slab &L, int s, double base, int lo, int hi,
                                        double rb)
{
    int step = 1;
    while (lo + step <= hi && sA(L, lo + step, s) - base <= rb) {
        lo += step;
        step <<= 1;
    }
    int top = min(hi, lo + step - 1);
    while (lo < top) {
        const int mid = (lo + top + 1) >> 1;
        if (sA(L, mid, s) - base <= rb) lo = mid;
        else top = mid - 1;
    }
    return lo;
}

// Compute-stream state of the walk.
struct Progress {
    int i;      // kernel in progress or next
    double w;   // unfinished fraction of kernel i
    double Ec;  // compute dynamic energy so far
};

// Advance compute in state s by at most `budget` seconds or up to the start of
// kernel `stop`.  Returns true when `stop` was reached; *el = time used.
__device__ inline bool advance(const Slab &L, Progress &g, int s, double budget, int stop,
                               double *el)
{
    double used = 0.0;
    if (g.w < 1.0) {
        const double need = g.w * sT(L, g.i, s);
        if (need <= budget) {
            g.Ec = g.Ec + sP(L, g.i, s) * need;
            used = need;
            g.i = g.i + 1;
            g.w = 1.0;
        } else {
            g.Ec = g.Ec + sP(L, g.i, s) * budget;
            g.w = g.w - budget / sT(L, g.i, s);
            if (g.w < 0.0) g.w = 0.0;
            *el = budget;
            return false;
        }
    }
    const double rb = budget - used;
    const int i0 = g.i;
    const double base = sA(L, i0, s);
    const int j = fit_from(L, s, base, i0, stop, rb);
    g.Ec = g.Ec + (sB(L, j, s) - sB(L, i0, s));
    if (j == stop) {
        *el = used + (sA(L, j, s) - base);
        g.i = j;
        return true;
    }
    const double r = rb - (sA(L, j, s) - base);
    g.Ec = g.Ec + sP(L, j, s) * r;
    g.w = 1.0 - r / sT(L, j, s);
    if (g.w < 0.0) g.w = 0.0;
    g.i = j;
    *el = budget;
    return false;
}

// General walk for M comm kernels (positions pos[], SM choices sm[]).
__device__ inline void cost_general(const Slab &L, int M, const int *pos, const int *sm,
                                    double p_static, double *T_out, double *E_out)
{
    Progress g{0, 1.0, 0.0};
    double tau = 0.0, el = 0.0, T = 0.0;
    bool finished = false;
    for (int m = 0; m < M; ++m) {
        const double tcm = L.tc[m * L.S + sm[m]];
        if (g.i < pos[m]) {
            advance(L, g, 0, INFINITY, pos[m], &el);
            tau = tau + el;
        }
        const double start = tau;
        if (advance(L, g, sm[m] + 1, tcm, L.N, &el)) {
            T = start + tcm;
            for (int q = m + 1; q < M; ++q) T = T + L.tc[q * L.S + sm[q]];
            finished = true;
            break;
        }
        tau = start + tcm;
    }
    if (!finished) {
        advance(L, g, 0, INFINITY, L.N, &el);
        T = tau + el;
    }
    double E = p_static * T;
    E = E + g.Ec;
    for (int m = 0; m < M; ++m) E = E + L.pc[m * L.S + sm[m]] * L.tc[m * L.S + sm[m]];
    *T_out = T;
    *E_out = E;
}

// One comm kernel launched with kernel p, SM choice s, whose comm phase ends inside
// kernel j (or at the end of compute when j == N): the same walk with the phases
// unrolled.  Compute first runs in state 0 up to kernel p (exactly A_0[p] seconds,
// B_0[p] joules); the comm phase covers kernels p..j-1 in state sigma and a fraction
// of kernel j; the rest runs in state 0.
__device__ __forceinline__ void cost_one_comm(const Slab &L, int p, int s, int j, double tcm,
                                              double pcm, double p_static, double *T_out,
                                              double *E_out)
{
    const int N = L.N, sg = s + 1;
    const double start = sA(L, p, 0);
    double Ec = sB(L, p, 0);
    Ec = Ec + (sB(L, j, sg) - sB(L, p, sg));
    double T;
    if (j == N) {
        T = start + tcm;
    } else {
        const double r = tcm - (sA(L, j, sg) - sA(L, p, sg));
        Ec = Ec + sP(L, j, sg) * r;
        double w = 1.0 - r / sT(L, j, sg);
        if (w < 0.0) w = 0.0;
        const double tau = start + tcm;
        double used = 0.0;
        int i = j;
        if (w < 1.0) {
            const double need = w * sT(L, j, 0);
            Ec = Ec + sP(L, j, 0) * need;
            used = need;
            i = j + 1;
        }
        Ec = Ec + (sB(L, N, 0) - sB(L, i, 0));
        const double el = used + (sA(L, N, 0) - sA(L, i, 0));
        T = tau + el;
    }
    double E = p_static * T;
    E = E + Ec;
    E = E + pcm * tcm;
    *T_out = T;
    *E_out = E;
}

__device__ __forceinline__ void eval_candidate(const Slab &L, const EvalArgs &a, int c,
                                               double *T, double *E)
{
    if (a.M == 1) {
        const int p = c / a.S, s = c - (c / a.S) * a.S;
        const double tcm = L.tc[s];
        const int j = fit_from(L, s + 1, sA(L, p, s + 1), p, L.N, tcm);
        cost_one_comm(L, p, s, j, tcm, L.pc[s], a.p_static, T, E);
    } else {
        const int SS = a.S * a.S;
        const int pp = c / SS, r = c - pp * SS;
        const int pr = L.pairs[pp];
        const int pos[2] = {pr & 0xFFFF, pr >> 16};
        const int sm[2] = {r / a.S, r % a.S};
        cost_general(L, 2, pos, sm, a.p_static, T, E);
    }
}

// Position-pair table (M = 2), once per block.
__device__ inline void build_pairs(const EvalArgs &a, int32_t *pairs)
{
    if (a.M != 2) return;
    for (int p1 = threadIdx.x; p1 < a.n_pos; p1 += KR_BLOCK) {
        const int base = p1 * a.n_pos - p1 * (p1 - 1) / 2;
        for (int p2 = p1; p2 < a.n_pos; ++p2) pairs[base + (p2 - p1)] = p1 | (p2 << 16);
    }
}

// Running sums of the staged slab: thread c < S1 forms A[.][c], thread S1 + c forms
// B[.][c], each left to right.  Loads are issued eight rows ahead of the additions.
__device__ inline void running_sums(const EvalArgs &a, double *lds)
{
    const int S1 = a.S + 1, N = a.N;
    const Slab L = slab_view(a, lds);
    double *A = (double *)L.A, *B = (double *)L.B;
    for (int c = threadIdx.x; c < 2 * S1; c += KR_BLOCK) {
        const bool isA = c < S1;
        const int s = isA ? c : c - S1;
        double *row = isA ? A : B;
        double acc = 0.0;
        row[s] = acc;
        for (int i0 = 0; i0 < N; i0 += 8) {
            double v[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int i = min(i0 + q, N - 1);
                v[q] = isA ? L.t[i * S1 + s] : (L.pw[i * S1 + s] * L.t[i * S1 + s]);
            }
#pragma unroll
            for (int q = 0; q < 8; ++q)
                if (i0 + q < N) {
                    acc = acc + v[q];
                    row[(i0 + q + 1) * S1 + s] = acc;
                }
        }
    }
}

// Element x of the staged part of slab (p, f): t, then pw, then tc, then pc.
__device__ __forceinline__ double slab_elem(const EvalArgs &a, size_t pf, int x)
{
    const int slab = a.N * (a.S + 1), ms = a.M * a.S;
    if (x < slab) return a.t[pf * slab + x];
    x -= slab;
    if (x < slab) return a.pw[pf * slab + x];
    x -= slab;
    if (x < ms) return a.tc[pf * ms + x];
    return a.pc[pf * ms + (x - ms)];
}

// ----------------------------------------------------------------------------
// Unfused: time and energy of every candidate to HBM.  One block per (p, f).
__global__ void __launch_bounds__(KR_BLOCK) eval_kernel(EvalArgs a)
{
    extern __shared__ double lds[];
    const int p = blockIdx.x / a.F, f = blockIdx.x % a.F;
    const size_t pf = (size_t)p * a.F + f;
    const int staged = 2 * a.N * (a.S + 1) + 2 * a.M * a.S;
    for (int x = threadIdx.x; x < staged; x += KR_BLOCK) lds[x] = slab_elem(a, pf, x);
    const Slab L = slab_view(a, lds);
    build_pairs(a, (int32_t *)L.pairs);
    __syncthreads();
    running_sums(a, lds);
    __syncthreads();
    const size_t base = (size_t)p * a.C + (size_t)f * a.Cf;
    for (int c = threadIdx.x; c < a.Cf; c += KR_BLOCK) {
        double T, E;
        eval_candidate(L, a, c, &T, &E);
        a.T_out[base + c] = T;
        a.E_out[base + c] = E;
    }
}

hipError_t launch_eval(const EvalArgs &a, hipStream_t st)
{
    const size_t lds = (size_t)a.lds_doubles * sizeof(double);
    hipLaunchKernelGGL(eval_kernel, dim3(a.P * a.F), dim3(KR_BLOCK), lds, st, a);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Fused: block (p, b) owns partition p and frequencies [b*fb, min(F, (b+1)*fb)).  Per
// frequency: stage the slab prefetched into registers, issue the next slab's loads,
// form the running sums, then per tile evaluate and append the tile's frontier to the
// block's output list.
// Register prefetch of one slab: PFT doubles per thread of t and of pw, one of tc/pc.
template <int PFT>
struct Prefetch {
    double t[PFT], pw[PFT], c[2];

    __device__ __forceinline__ void load(const EvalArgs &a, size_t pf)
    {
        const int slab = a.N * (a.S + 1), ms = a.M * a.S;
        const double *gt = a.t + pf * slab, *gp = a.pw + pf * slab;
#pragma unroll
        for (int k = 0; k < PFT; ++k) {
            const int x = threadIdx.x + k * KR_BLOCK;
            if (x < slab) {
                t[k] = gt[x];
                pw[k] = gp[x];
            }
        }
        const int x = threadIdx.x;
        if (x < ms) {
            c[0] = a.tc[pf * ms + x];
            c[1] = a.pc[pf * ms + x];
        }
    }

    __device__ __forceinline__ void store(const EvalArgs &a, double *lds) const
    {
        const int slab = a.N * (a.S + 1), ms = a.M * a.S;
#pragma unroll
        for (int k = 0; k < PFT; ++k) {
            const int x = threadIdx.x + k * KR_BLOCK;
            if (x < slab) {
                lds[x] = t[k];
                lds[slab + x] = pw[k];
            }
        }
        const int x = threadIdx.x;
        if (x < ms) {
            lds[2 * slab + x] = c[0];
            lds[2 * slab + ms + x] = c[1];
        }
    }
};

template <int PFT, int CPT, bool ONE_COMM>
__global__ void __launch_bounds__(KR_BLOCK) eval_filter_kernel(EvalArgs a, UnitOut o)
{
    extern __shared__ double lds[];
    __shared__ FilterShared fsh;
    const int p = blockIdx.x / a.nfb, b = blockIdx.x % a.nfb;
    const int f0 = b * a.fb, f1 = min(a.F, f0 + a.fb);
    const Slab L = slab_view(a, lds);
    FilterLds fl;
    fl.sh = &fsh;
    fl.sT = (uint64_t *)(lds + a.surv_off);
    fl.sE = fl.sT + KR_SURV_CAP;
    fl.sI = (int32_t *)(fl.sE + KR_SURV_CAP);
    build_pairs(a, (int32_t *)L.pairs);

    Prefetch<PFT> pre;
    pre.load(a, (size_t)p * a.F + f0);
    const size_t slot0 = (size_t)p * a.C + (size_t)f0 * a.Cf;
    double *oT = o.T + slot0, *oE = o.E + slot0;
    int32_t *oI = o.I + slot0;
    int count = 0, parity = 0;
    // position runs of the one-comm mapping: thread = (SM choice s, run of cpt positions)
    const int s_of = threadIdx.x % a.S, run = threadIdx.x / a.S;

    for (int f = f0; f < f1; ++f) {
        lds_barrier();  // the previous slab is no longer read
        pre.store(a, lds);
        if (f + 1 < f1) pre.load(a, (size_t)p * a.F + f + 1);
        lds_barrier();
        running_sums(a, lds);
        lds_barrier();

        for (int tile = 0; tile < a.ntiles; ++tile) {
            double vT[CPT], vE[CPT];
            int32_t vI[CPT];
            bool ok[CPT];
            if (ONE_COMM) {
                // consecutive launch positions of one SM choice: the end-of-comm kernel
                // index j never decreases with the launch position
                const int s = s_of, sg = s_of + 1;
                const double tcm = L.tc[s], pcm = L.pc[s];
                const int pb = (tile * a.nchunk + run) * a.cpt;
                const bool live = run < a.nchunk;
                int j = 0;
#pragma unroll
                for (int k = 0; k < CPT; ++k) {
                    const int pos = pb + k;
                    ok[k] = live && k < a.cpt && pos < a.n_pos;
                    vT[k] = 0.0;
                    vE[k] = 0.0;
                    vI[k] = f * a.Cf + pos * a.S + s;
                    if (ok[k]) {
                        j = max(j, pos);
                        j = fit_from(L, sg, sA(L, pos, sg), j, a.N, tcm);
                        cost_one_comm(L, pos, s, j, tcm, pcm, a.p_static, &vT[k], &vE[k]);
                    }
                }
            } else {
                const int c0 = tile * a.tile;
                const int c1 = min(a.Cf, c0 + a.tile);
#pragma unroll
                for (int k = 0; k < CPT; ++k) {
                    const int c = c0 + threadIdx.x + k * KR_BLOCK;
                    ok[k] = k < a.cpt && c < c1;
                    vT[k] = 0.0;
                    vE[k] = 0.0;
                    vI[k] = f * a.Cf + c;
                    if (ok[k]) eval_candidate(L, a, c, &vT[k], &vE[k]);
                }
            }
            count += tile_frontier<CPT>(vT, vE, vI, ok, fl, parity, oT + count, oE + count,
                                        oI + count);
        }
    }
    if (threadIdx.x == 0) o.cnt[blockIdx.x] = count;
}

template <int PFT, int CPT>
static void launch_ef3(const EvalArgs &a, const UnitOut &o, size_t lds, hipStream_t st)
{
    const dim3 grid(a.P * a.nfb), block(KR_BLOCK);
    if (a.one_comm)
        hipLaunchKernelGGL((eval_filter_kernel<PFT, CPT, true>), grid, block, lds, st, a, o);
    else
        hipLaunchKernelGGL((eval_filter_kernel<PFT, CPT, false>), grid, block, lds, st, a, o);
}

template <int PFT>
static void launch_ef2(const EvalArgs &a, const UnitOut &o, size_t lds, hipStream_t st)
{
    if (a.cpt <= 2) launch_ef3<PFT, 2>(a, o, lds, st);
    else if (a.cpt <= 5) launch_ef3<PFT, 5>(a, o, lds, st);
    else launch_ef3<PFT, 8>(a, o, lds, st);
}

hipError_t launch_eval_filter(const EvalArgs &a, const UnitOut &o, hipStream_t st)
{
    const size_t lds = (size_t)a.lds_doubles * sizeof(double);
    if (a.pf <= 2) launch_ef2<2>(a, o, lds, st);
    else if (a.pf <= 5) launch_ef2<5>(a, o, lds, st);
    else if (a.pf <= 8) launch_ef2<8>(a, o, lds, st);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// Candidate index -> (f, positions, SM choices).
__global__ void decode_kernel(DecodeArgs d)
{
    const int64_t q = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x;
    if (q >= d.n) return;
    int c = d.idx[q];
    const int Cf = d.Cf;
    if (c < 0 || c >= Cf * d.F) {
        d.f_out[q] = -1;
        for (int m = 0; m < d.M; ++m) d.pos_out[q * d.M + m] = d.sm_out[q * d.M + m] = -1;
        return;
    }
    const int f = c / Cf;
    c -= f * Cf;
    d.f_out[q] = f;
    if (d.M == 1) {
        d.pos_out[q] = c / d.S;
        d.sm_out[q] = c % d.S;
        return;
    }
    const int SS = d.S * d.S;
    int pp = c / SS;
    const int r = c - pp * SS;
    int p1 = 0;
    while (pp >= d.n_pos - p1) {
        pp -= d.n_pos - p1;
        ++p1;
    }
    d.pos_out[q * 2] = p1;
    d.pos_out[q * 2 + 1] = p1 + pp;
    d.sm_out[q * 2] = r / d.S;
    d.sm_out[q * 2 + 1] = r % d.S;
}

hipError_t launch_decode(const DecodeArgs &d, hipStream_t st)
{
    if (d.n == 0) return hipSuccess;
    hipLaunchKernelGGL(decode_kernel, dim3((unsigned)((d.n + KR_BLOCK - 1) / KR_BLOCK)),
                       dim3(KR_BLOCK), 0, st, d);
    return hipGetLastError();
}

}  // namespace kr
