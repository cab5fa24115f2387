// Candidate evaluation on gfx950.
//
// One workgroup per (partition, frequency).  The (kernel x SM-state) slab of the time
// and power tables for that frequency is contiguous in HBM; it is staged into LDS
// with coalesced loads, the per-state running sums of time and energy are formed in
// LDS (one thread per state column, left to right), and then one thread per
// candidate walks the partition cost model reading only LDS.
//
// Cost model (fluid SM-share reading of Sections 3.2 and 4.2; the paper gives no
// closed form, Section 4.3.1): compute kernels progress at 1/t in the current SM
// state; comm kernel m is launched when compute reaches the start of kernel p_m and
// starts when the comm stream is free (FIFO); while it runs, compute is in state
// s_m + 1.  T = later of compute end and last comm end; E = p_static * T + compute
// dynamic energy + comm dynamic energy (Sections 2.1, 2.3, 4.5).  Every line below
// is one IEEE fp64 rounding in a fixed order; the library is built without FMA
// contraction so the results are reproducible bit for bit.
#include "kr_launch.h"
#include "kr_tile.h"

namespace kr {

// LDS slab of one (partition, frequency).
struct Slab {
    const double *t;   // [N][S1] kernel time per state
    const double *pw;  // [N][S1] kernel dynamic power per state
    const double *A;   // [S1][N+1] running sums of t, left to right
    const double *B;   // [S1][N+1] running sums of pw*t
    const double *tc;  // [M][S]
    const double *pc;  // [M][S]
    const int32_t *pairs;  // [n_pp] p1 | p2 << 16 (M = 2)
    int N, S1, S;
};

__device__ __forceinline__ double sA(const Slab &L, int s, int i) { return L.A[s * (L.N + 1) + i]; }
__device__ __forceinline__ double sB(const Slab &L, int s, int i) { return L.B[s * (L.N + 1) + i]; }
__device__ __forceinline__ double sT(const Slab &L, int i, int s) { return L.t[i * L.S1 + s]; }
__device__ __forceinline__ double sP(const Slab &L, int i, int s) { return L.pw[i * L.S1 + s]; }

// Largest j in [i0, stop] with A[s][j] - A[s][i0] <= rb (the predicate is monotone
// in j because the running sums never decrease).
__device__ __forceinline__ int fit_kernels(const Slab &L, int s, int i0, int stop, double rb)
{
    const double base = sA(L, s, i0);
    int lo = i0, hi = stop;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (sA(L, s, mid) - base <= rb) lo = mid;
        else hi = mid - 1;
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
        double need = g.w * sT(L, g.i, s);
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
    const int j = fit_kernels(L, s, i0, stop, rb);
    g.Ec = g.Ec + (sB(L, s, j) - sB(L, s, i0));
    if (j == stop) {
        *el = used + (sA(L, s, j) - sA(L, s, i0));
        g.i = j;
        return true;
    }
    const double r = rb - (sA(L, s, j) - sA(L, s, i0));
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

// One comm kernel: the same walk with the phases unrolled.  Compute first runs in
// state 0 up to kernel p (exactly A_0[p] seconds, B_0[p] joules); the comm phase then
// covers whole kernels p..j-1 in state sigma and a fraction of kernel j; the rest
// runs in state 0.
__device__ __forceinline__ void cost_one_comm(const Slab &L, int p, int s, double p_static,
                                              double *T_out, double *E_out)
{
    const int N = L.N, sg = s + 1;
    const double tcm = L.tc[s], pcm = L.pc[s];
    const double start = sA(L, 0, p);
    double Ec = sB(L, 0, p);
    const int j = fit_kernels(L, sg, p, N, tcm);
    Ec = Ec + (sB(L, sg, j) - sB(L, sg, p));
    double T;
    if (j == N) {
        T = start + tcm;
    } else {
        const double r = tcm - (sA(L, sg, j) - sA(L, sg, p));
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
        Ec = Ec + (sB(L, 0, N) - sB(L, 0, i));
        const double el = used + (sA(L, 0, N) - sA(L, 0, i));
        T = tau + el;
    }
    double E = p_static * T;
    E = E + Ec;
    E = E + pcm * tcm;
    *T_out = T;
    *E_out = E;
}

// Stage the slab of (partition p, frequency f) and form the running sums.
__device__ inline Slab stage_slab(const EvalArgs &a, int p, int f, double *lds, int32_t *ldsi)
{
    const int N = a.N, S = a.S, S1 = S + 1, M = a.M;
    double *t = lds;
    double *pw = t + N * S1;
    double *A = pw + N * S1;
    double *B = A + S1 * (N + 1);
    double *tc = B + S1 * (N + 1);
    double *pc = tc + M * S;
    const size_t slab = (size_t)N * S1;
    const size_t pf = (size_t)p * a.F + f;
    const double *gt = a.t + pf * slab;
    const double *gp = a.pw + pf * slab;
    for (int x = threadIdx.x; x < (int)slab; x += KR_BLOCK) {
        t[x] = gt[x];
        pw[x] = gp[x];
    }
    const double *gtc = a.tc + pf * (size_t)(M * S);
    const double *gpc = a.pc + pf * (size_t)(M * S);
    for (int x = threadIdx.x; x < M * S; x += KR_BLOCK) {
        tc[x] = gtc[x];
        pc[x] = gpc[x];
    }
    if (M == 2) {
        for (int p1 = threadIdx.x; p1 < a.n_pos; p1 += KR_BLOCK) {
            const int base = p1 * a.n_pos - p1 * (p1 - 1) / 2;
            for (int p2 = p1; p2 < a.n_pos; ++p2) ldsi[base + (p2 - p1)] = p1 | (p2 << 16);
        }
    }
    __syncthreads();
    for (int c = threadIdx.x; c < 2 * S1; c += KR_BLOCK) {
        const int s = c < S1 ? c : c - S1;
        double *row = (c < S1 ? A : B) + s * (N + 1);
        double acc = 0.0;
        row[0] = acc;
        if (c < S1) {
            for (int i = 0; i < N; ++i) {
                acc = acc + t[i * S1 + s];
                row[i + 1] = acc;
            }
        } else {
            for (int i = 0; i < N; ++i) {
                acc = acc + (pw[i * S1 + s] * t[i * S1 + s]);
                row[i + 1] = acc;
            }
        }
    }
    __syncthreads();
    return Slab{t, pw, A, B, tc, pc, ldsi, N, S1, S};
}

__device__ __forceinline__ void eval_candidate(const Slab &L, const EvalArgs &a, int c,
                                               double *T, double *E)
{
    if (a.M == 1) {
        cost_one_comm(L, c / a.S, c % a.S, a.p_static, T, E);
    } else {
        const int SS = a.S * a.S;
        const int pp = c / SS, r = c - pp * SS;
        const int pr = L.pairs[pp];
        int pos[2] = {pr & 0xFFFF, pr >> 16};
        int sm[2] = {r / a.S, r % a.S};
        cost_general(L, 2, pos, sm, a.p_static, T, E);
    }
}

__global__ void __launch_bounds__(KR_BLOCK) eval_kernel(EvalArgs a)
{
    extern __shared__ double lds[];
    const int p = blockIdx.x / a.F, f = blockIdx.x % a.F;
    int32_t *ldsi = (int32_t *)(lds + a.slab_doubles);
    const Slab L = stage_slab(a, p, f, lds, ldsi);
    const size_t base = (size_t)p * a.C + (size_t)f * a.Cf;
    for (int c = threadIdx.x; c < a.Cf; c += KR_BLOCK) {
        double T, E;
        eval_candidate(L, a, c, &T, &E);
        a.T_out[base + c] = T;
        a.E_out[base + c] = E;
    }
}

template <int CPT>
__global__ void __launch_bounds__(KR_BLOCK) eval_filter_kernel(EvalArgs a, TileOut o)
{
    extern __shared__ double lds[];
    __shared__ TileScratch sc;
    const int p = blockIdx.x / a.F, f = blockIdx.x % a.F;
    int32_t *ldsi = (int32_t *)(lds + a.slab_doubles);
    const Slab L = stage_slab(a, p, f, lds, ldsi);
    uint64_t *tile_mem = (uint64_t *)(lds + a.slab_doubles + a.pair_doubles);
    TileLds tl;
    tl.nb = o.nb;
    tl.cap = a.tile;
    tl.bkt = tile_mem;
    tl.sT = tl.bkt + o.nb;
    tl.sE = tl.sT + a.tile;
    tl.sI = (int32_t *)(tl.sE + a.tile);
    const int ntf = a.tiles_per_freq;
    for (int sub = 0; sub < ntf; ++sub) {
        const int c0 = sub * a.tile;
        const int c1 = min(a.Cf, c0 + a.tile);
        double vT[CPT], vE[CPT];
        int32_t vI[CPT];
        bool ok[CPT];
#pragma unroll
        for (int k = 0; k < CPT; ++k) {
            const int c = c0 + threadIdx.x + k * KR_BLOCK;
            ok[k] = c < c1;
            vT[k] = 0.0;
            vE[k] = 0.0;
            vI[k] = f * a.Cf + c;
            if (ok[k]) eval_candidate(L, a, c, &vT[k], &vE[k]);
        }
        const size_t slot = (size_t)p * a.C + (size_t)f * a.Cf + c0;
        const int n = tile_frontier<CPT>(vT, vE, vI, ok, tl, sc, o.T + slot, o.E + slot,
                                         o.I + slot);
        if (threadIdx.x == 0) o.cnt[(size_t)p * o.tiles_per_seg + f * ntf + sub] = n;
    }
}

hipError_t launch_eval(const EvalArgs &a, hipStream_t st)
{
    const size_t lds = (size_t)(a.slab_doubles + a.pair_doubles) * sizeof(double);
    hipLaunchKernelGGL(eval_kernel, dim3(a.P * a.F), dim3(KR_BLOCK), lds, st, a);
    return hipGetLastError();
}

hipError_t launch_eval_filter(const EvalArgs &a, const TileOut &o, hipStream_t st)
{
    const size_t lds = (size_t)(a.slab_doubles + a.pair_doubles) * sizeof(double) +
                       (size_t)o.nb * 8 + (size_t)a.tile * 20;
    const dim3 grid(a.P * a.F), block(KR_BLOCK);
    switch (a.cpt) {
    case 1: hipLaunchKernelGGL(eval_filter_kernel<1>, grid, block, lds, st, a, o); break;
    case 2: hipLaunchKernelGGL(eval_filter_kernel<2>, grid, block, lds, st, a, o); break;
    case 4: hipLaunchKernelGGL(eval_filter_kernel<4>, grid, block, lds, st, a, o); break;
    case 5: hipLaunchKernelGGL(eval_filter_kernel<5>, grid, block, lds, st, a, o); break;
    default: hipLaunchKernelGGL(eval_filter_kernel<8>, grid, block, lds, st, a, o); break;
    }
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
