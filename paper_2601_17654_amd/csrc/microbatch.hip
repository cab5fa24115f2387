// Microbatch frontier (Section 4.4, Algorithm 2 with one GPU frequency per microbatch and
// one shared configuration per partition type).  The host entry point composes each
// frequency's scaled type frontiers with the frontier composition, then these kernels
// walk every non-dominated bin back to its configuration, sum it exactly in execution
// order, and hand the union over frequencies to GetFrontier.
#include "kr_launch.h"
#include "kr_device.h"

namespace kr {

// Points of the used types at frequency f, scaled by their repeat counts, in type order:
// off_f [Ku + 1], Ts, Es.  One block.
__global__ void __launch_bounds__(KR_BLOCK) mb_scale_kernel(MbArgs a, int f, int64_t *off_f,
                                                          double *Ts, double *Es)
{
    __shared__ int64_t so[KR_MB_MAX_TYPES + 1];
    if (threadIdx.x == 0) {
        int64_t w = 0;
        for (int u = 0; u < a.Ku; ++u) {
            so[u] = w;
            const int t = a.used[u];
            w += a.seg_off[t * a.F + f + 1] - a.seg_off[t * a.F + f];
        }
        so[a.Ku] = w;
    }
    __syncthreads();
    for (int u = threadIdx.x; u <= a.Ku; u += KR_BLOCK) off_f[u] = so[u];
    for (int u = 0; u < a.Ku; ++u) {
        const int t = a.used[u];
        const int64_t lo = a.seg_off[t * a.F + f], n = so[u + 1] - so[u];
        const double m = (double)a.count[u];
        for (int64_t j = threadIdx.x; j < n; j += KR_BLOCK) {
            Ts[so[u] + j] = m * a.T[lo + j];
            Es[so[u] + j] = m * a.E[lo + j];
        }
    }
}

// Slot f * B + q of the union: the configuration behind frequency f's q-th non-dominated
// bin, or +inf when there is none (q past the staircase, or the composition failed).
__global__ void __launch_bounds__(KR_BLOCK) mb_walk_kernel(MbArgs a, int f, MbComp c)
{
    const int q = blockIdx.x * KR_BLOCK + threadIdx.x;
    if (q >= a.B) return;
    const int64_t slot = (int64_t)f * a.B + q;
    int32_t *ch = a.slot_choice + slot * a.K;
    const bool live = *c.status == KR_OK && q < *c.n_stair;
    int32_t choice[KR_MB_MAX_TYPES];
    bool ok = live;
    if (ok) {
        int64_t b = c.stair_bin[q];
        for (int u = a.Ku - 1; u >= 0 && ok; --u) {
            const int32_t j = c.bp[(int64_t)u * a.B + b];
            ok = j >= 0;
            choice[u] = j;
            if (ok) b -= c.pt_bin[c.off[u] + j];
        }
        ok = ok && b == 0;
    }
    if (!ok) {
        a.slot_T[slot] = INFINITY;
        a.slot_E[slot] = INFINITY;
        for (int t = 0; t < a.K; ++t) ch[t] = -1;
        return;
    }
    // exact sums: partitions in execution order, then the components
    double Tm = 0.0, Em = 0.0;
    for (int i = 0; i < a.n_seq; ++i) {
        const int u = a.seq_u[i];
        const int64_t x = a.seg_off[a.used[u] * a.F + f] + choice[u];
        Tm = Tm + a.T[x];
        Em = Em + a.E[x];
    }
    for (int k = 0; k < a.n_comp; ++k) {
        Tm = Tm + a.comp_T[(int64_t)k * a.F + f];
        Em = Em + a.comp_E[(int64_t)k * a.F + f];
    }
    a.slot_T[slot] = Tm;
    a.slot_E[slot] = Em;
    for (int t = 0; t < a.K; ++t) ch[t] = -1;
    for (int u = 0; u < a.Ku; ++u) ch[a.used[u]] = choice[u];
}

__global__ void mb_seg_kernel(int64_t *seg, int64_t n)
{
    if (threadIdx.x == 0) {
        seg[0] = 0;
        seg[1] = n;
    }
}

// Frontier points (slot indices from GetFrontier) into the caller's outputs.
__global__ void __launch_bounds__(KR_BLOCK) mb_gather_kernel(MbArgs a, const int64_t *front_off,
                                                           const int32_t *front_idx, int64_t cap,
                                                           double *out_T, double *out_E,
                                                           int32_t *out_f, int32_t *out_choice,
                                                           int64_t *n_out)
{
    const int64_t n = front_off[1];
    const int64_t r = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x;
    if (r == 0) *n_out = n;
    if (r >= n || r >= cap) return;
    const int64_t slot = front_idx[r];
    out_T[r] = a.slot_T[slot];
    out_E[r] = a.slot_E[slot];
    out_f[r] = (int32_t)(slot / a.B);
    for (int t = 0; t < a.K; ++t) out_choice[r * a.K + t] = a.slot_choice[slot * a.K + t];
}

hipError_t launch_mb_scale(const MbArgs &a, int f, int64_t *off_f, double *Ts, double *Es,
                           hipStream_t st)
{
    hipLaunchKernelGGL(mb_scale_kernel, dim3(1), dim3(KR_BLOCK), 0, st, a, f, off_f, Ts, Es);
    return hipGetLastError();
}

hipError_t launch_mb_walk(const MbArgs &a, int f, const MbComp &c, hipStream_t st)
{
    hipLaunchKernelGGL(mb_walk_kernel, dim3((a.B + KR_BLOCK - 1) / KR_BLOCK), dim3(KR_BLOCK), 0,
                       st, a, f, c);
    return hipGetLastError();
}

hipError_t launch_mb_seg(int64_t *seg, int64_t n, hipStream_t st)
{
    hipLaunchKernelGGL(mb_seg_kernel, dim3(1), dim3(64), 0, st, seg, n);
    return hipGetLastError();
}

hipError_t launch_mb_gather(const MbArgs &a, const int64_t *front_off, const int32_t *front_idx,
                            int64_t cap, double *out_T, double *out_E, int32_t *out_f,
                            int32_t *out_choice, int64_t *n_out, hipStream_t st)
{
    const int64_t n = (int64_t)a.F * a.B;
    const int64_t m = cap < n ? cap : n;
    const int64_t blocks = (m > 0 ? m : 1) + KR_BLOCK - 1;
    hipLaunchKernelGGL(mb_gather_kernel, dim3((unsigned)(blocks / KR_BLOCK)), dim3(KR_BLOCK), 0, st,
                       a, front_off, front_idx, cap, out_T, out_E, out_f, out_choice, n_out);
    return hipGetLastError();
}

// ---- enumeration of every configuration (Algorithm 2 as written) ----------------------

// Configurations per frequency (product of the used types' point counts) and their
// running totals: base[f] .. base[f+1]-1 are frequency f's slots.  One thread; fails
// with KR_ECAPACITY past the slots reserved.
__global__ void mb_count_kernel(MbArgs a, int64_t *base, int64_t slots, int32_t *status)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int64_t tot = 0;
    for (int f = 0; f < a.F; ++f) {
        base[f] = tot;
        int64_t n = 1;
        for (int u = 0; u < a.Ku; ++u) {
            const int t = a.used[u];
            n *= a.seg_off[t * a.F + f + 1] - a.seg_off[t * a.F + f];
        }
        tot += n;
    }
    base[a.F] = tot;
    *status = tot <= slots ? KR_OK : KR_ECAPACITY;
}

// Frequency and per-used-type point of slot x (first used type slowest).
__device__ __forceinline__ int mb_decode(const MbArgs &a, const int64_t *base, int64_t x,
                                         int32_t *choice)
{
    int lo = 0, hi = a.F - 1;  // last f with base[f] <= x
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (base[mid] <= x) lo = mid;
        else hi = mid - 1;
    }
    const int f = lo;
    int64_t c = x - base[f];
    for (int u = a.Ku - 1; u >= 0; --u) {
        const int t = a.used[u];
        const int64_t n = a.seg_off[t * a.F + f + 1] - a.seg_off[t * a.F + f];
        choice[u] = (int32_t)(c % n);
        c /= n;
    }
    return f;
}

// Time and energy of every configuration: partitions in execution order, then the
// components.  Slots past the total hold +inf.
__global__ void __launch_bounds__(KR_BLOCK) mb_enum_kernel(MbArgs a, const int64_t *base,
                                                         int64_t slots, const int32_t *status)
{
    const int64_t total = *status == KR_OK ? base[a.F] : 0;
    for (int64_t x = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x; x < slots;
         x += (int64_t)gridDim.x * KR_BLOCK) {
        if (x >= total) {
            a.slot_T[x] = INFINITY;
            a.slot_E[x] = INFINITY;
            continue;
        }
        int32_t choice[KR_MB_MAX_TYPES];
        const int f = mb_decode(a, base, x, choice);
        double Tm = 0.0, Em = 0.0;
        for (int i = 0; i < a.n_seq; ++i) {
            const int u = a.seq_u[i];
            const int64_t p = a.seg_off[a.used[u] * a.F + f] + choice[u];
            Tm = Tm + a.T[p];
            Em = Em + a.E[p];
        }
        for (int k = 0; k < a.n_comp; ++k) {
            Tm = Tm + a.comp_T[(int64_t)k * a.F + f];
            Em = Em + a.comp_E[(int64_t)k * a.F + f];
        }
        a.slot_T[x] = Tm;
        a.slot_E[x] = Em;
    }
}

// Frontier slots into the caller's outputs, decoding each slot's configuration.
__global__ void __launch_bounds__(KR_BLOCK) mb_enum_gather_kernel(
    MbArgs a, const int64_t *base, const int32_t *status, const int64_t *front_off,
    const int32_t *front_idx, int64_t cap, double *out_T, double *out_E, int32_t *out_f,
    int32_t *out_choice, int64_t *n_out)
{
    const int64_t n = *status == KR_OK ? front_off[1] : 0;
    const int64_t r = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x;
    if (r == 0) *n_out = n;
    if (r >= n || r >= cap) return;
    const int64_t x = front_idx[r];
    int32_t choice[KR_MB_MAX_TYPES];
    const int f = mb_decode(a, base, x, choice);
    out_T[r] = a.slot_T[x];
    out_E[r] = a.slot_E[x];
    out_f[r] = f;
    for (int t = 0; t < a.K; ++t) out_choice[r * a.K + t] = -1;
    for (int u = 0; u < a.Ku; ++u) out_choice[r * a.K + a.used[u]] = choice[u];
}

hipError_t launch_mb_enum(const MbArgs &a, int64_t *base, int64_t slots, int32_t *status,
                          hipStream_t st)
{
    hipLaunchKernelGGL(mb_count_kernel, dim3(1), dim3(64), 0, st, a, base, slots, status);
    const int64_t blocks = (slots + KR_BLOCK - 1) / KR_BLOCK;
    const unsigned grid = (unsigned)(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096);
    hipLaunchKernelGGL(mb_enum_kernel, dim3(grid), dim3(KR_BLOCK), 0, st, a, base, slots,
                       (const int32_t *)status);
    return hipGetLastError();
}

hipError_t launch_mb_enum_gather(const MbArgs &a, const int64_t *base, const int32_t *status,
                                 const int64_t *front_off, const int32_t *front_idx, int64_t cap,
                                 double *out_T, double *out_E, int32_t *out_f, int32_t *out_choice,
                                 int64_t *n_out, int64_t slots, hipStream_t st)
{
    const int64_t m = cap < slots ? cap : slots;
    const int64_t blocks = ((m > 0 ? m : 1) + KR_BLOCK - 1) / KR_BLOCK;
    hipLaunchKernelGGL(mb_enum_gather_kernel, dim3((unsigned)blocks), dim3(KR_BLOCK), 0, st, a,
                       base, status, front_off, front_idx, cap, out_T, out_E, out_f, out_choice,
                       n_out);
    return hipGetLastError();
}

}  // namespace kr
