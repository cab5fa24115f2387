// Frontier composition (Section 4.4, Algorithm 2) and schedule extraction
// (Section 5.1).
//
// Algorithm 2 sums time and energy over every one-point-per-partition choice and
// keeps the frontier.  Here time is discretised: with bin width delta, point j of
// partition k sits at offset floor((T_j - tmin_k) / delta); e_k[b] is the least
// energy at offset b, and
//     F_1 = e_1,   F_k[b] = min_{b2} F_{k-1}[b - b2] + e_k[b2]
// is a min-plus convolution, one partition at a time.  Back-pointers record the point
// chosen for partition k at each composite bin, so any composed bin can be walked
// back to its per-partition choice.  Ties: e_k keeps the smallest point index, the
// min-plus keeps the smallest b2 (strict comparisons in ascending order).
#include "kr_launch.h"
#include "kr_device.h"

namespace kr {

struct MinF64 {
    __device__ __forceinline__ double operator()(double a, double b) const { return b < a ? b : a; }
};
struct MaxF64 {
    __device__ __forceinline__ double operator()(double a, double b) const { return b > a ? b : a; }
};

__device__ __forceinline__ uint64_t load_l2(const uint64_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t load_l2(const int32_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void compose_init_kernel(ComposeArgs a)
{
    if (threadIdx.x == 0) *a.status = KR_OK;
}

// Per-partition time range.
__global__ void __launch_bounds__(KR_BLOCK) compose_range_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ double sc[KR_WAVES];
    const int k = blockIdx.x;
    const int64_t lo = a.off[k], hi = a.off[k + 1];
    if (hi <= lo) {
        if (threadIdx.x == 0) *a.status = KR_EINVAL;
        return;
    }
    double mn = INFINITY, mx = -INFINITY;
    for (int64_t j = lo + threadIdx.x; j < hi; j += KR_BLOCK) {
        const double t = a.T[j];
        mn = t < mn ? t : mn;
        mx = t > mx ? t : mx;
    }
    mn = block_reduce(mn, (double)INFINITY, MinF64(), sc);
    mx = block_reduce(mx, -(double)INFINITY, MaxF64(), sc);
    if (threadIdx.x == 0) {
        w.tmin[k] = mn;
        w.range[k] = mx - mn;
    }
}

// Bin width, per-partition bin counts and running bin totals (sequential sums, in
// partition order, so the width is reproducible bit for bit).
__global__ void compose_setup_kernel(ComposeArgs a, ComposeWs w)
{
    if (threadIdx.x != 0 || *a.status != KR_OK) return;
    const int P = a.P, B = a.B;
    double R = 0.0;
    for (int k = 0; k < P; ++k) R = R + w.range[k];
    double delta;
    if (a.delta_in > 0.0) delta = a.delta_in;
    else if (R > 0.0) delta = R / (double)(B - 1);
    else delta = 1.0;
    for (int iter = 0;; ++iter) {
        int64_t total = 1;
        for (int k = 0; k < P; ++k) {
            const double x = floor(w.range[k] / delta);
            const int64_t m = x < (double)B ? (int64_t)x : (int64_t)B;
            w.Mk[k] = m;
            total += m;
        }
        if (total <= B) break;
        if (a.delta_in > 0.0 || iter > 4096) {
            *a.status = KR_ECAPACITY;
            return;
        }
        delta = __longlong_as_double(__double_as_longlong(delta) + 1);  // next double up
    }
    double tmin_sum = 0.0;
    for (int k = 0; k < P; ++k) tmin_sum = tmin_sum + w.tmin[k];
    int64_t L = 0, e = 0;
    for (int k = 0; k < P; ++k) {
        L = (k == 0) ? w.Mk[0] + 1 : L + w.Mk[k];
        w.Lk[k] = L;
        w.eoff[k] = e;
        e += w.Mk[k] + 1;
    }
    w.eoff[P] = e;
    a.info[0] = delta;
    a.info[1] = tmin_sum;
    *a.L_out = (int32_t)L;
}

// Offsets of every point, least energy per offset, and the list of occupied offsets.
__global__ void __launch_bounds__(KR_BLOCK) compose_bin_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ int32_t sc[KR_WAVES];
    if (*a.status != KR_OK) return;
    const int k = blockIdx.x;
    const int64_t lo = a.off[k], hi = a.off[k + 1];
    const int64_t M = w.Mk[k], eo = w.eoff[k];
    const double tmin = w.tmin[k], delta = a.info[0];
    uint64_t *eb = w.ebits + eo;
    int32_t *ea = w.earg + eo;
    for (int64_t b = threadIdx.x; b <= M; b += KR_BLOCK) {
        eb[b] = KR_INF_BITS;
        ea[b] = 0x7FFFFFFF;
    }
    __syncthreads();
    for (int64_t j = lo + threadIdx.x; j < hi; j += KR_BLOCK) {
        const double x = floor((a.T[j] - tmin) / delta);
        const int64_t o = !(x > 0.0) ? 0 : (x < (double)M ? (int64_t)x : M);
        a.pt_bin[j] = (int32_t)o;
        atomicMin((unsigned long long *)&eb[o], (unsigned long long)dbits(a.E[j]));
    }
    __syncthreads();
    for (int64_t j = lo + threadIdx.x; j < hi; j += KR_BLOCK) {
        const int32_t o = a.pt_bin[j];
        if (dbits(a.E[j]) == load_l2(&eb[o])) atomicMin(&ea[o], (int32_t)(j - lo));
    }
    __syncthreads();
    int32_t carry = 0;
    for (int64_t b0 = 0; b0 <= M; b0 += KR_BLOCK) {
        const int64_t b = b0 + threadIdx.x;
        const int32_t arg = b <= M ? load_l2(&ea[b]) : 0x7FFFFFFF;
        const int has = arg != 0x7FFFFFFF;
        int32_t tot;
        const int32_t pos = block_exclusive(has, 0, SumI32(), sc, &tot);
        if (has) {
            w.ob2[eo + carry + pos] = (int32_t)b;
            w.oe[eo + carry + pos] = bitsd(load_l2(&eb[b]));
            w.oarg[eo + carry + pos] = arg;
        }
        carry += tot;
    }
    if (threadIdx.x == 0) w.occ[k] = carry;
}

// F_1 and the first row of back-pointers.
__global__ void compose_first_kernel(ComposeArgs a, ComposeWs w, double *F)
{
    if (*a.status != KR_OK) return;
    const int64_t b = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x;
    if (b >= a.B) return;
    double v = INFINITY;
    int32_t who = -1;
    if (b <= w.Mk[0]) {
        const int32_t arg = w.earg[b];
        if (arg != 0x7FFFFFFF) {
            v = bitsd(w.ebits[b]);
            who = arg;
        }
    }
    F[b] = v;
    a.bp[b] = who;
}

// One min-plus step: F_k[b] = min over occupied b2 of F_{k-1}[b - b2] + e_k[b2].
__global__ void __launch_bounds__(KR_BLOCK)
minplus_step_kernel(ComposeArgs a, ComposeWs w, int k, const double *Fprev, double *Fcur)
{
    __shared__ int32_t sb2[KR_BLOCK], sarg[KR_BLOCK];
    __shared__ double se[KR_BLOCK];
    if (*a.status != KR_OK) return;
    const int64_t b = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x;
    const int64_t Lprev = w.Lk[k - 1], Lcur = w.Lk[k];
    const int cnt = w.occ[k];
    const int64_t base = w.eoff[k];
    double best = INFINITY;
    int32_t who = -1;
    const bool live = b < Lcur;
    for (int c0 = 0; c0 < cnt; c0 += KR_BLOCK) {
        const int q = c0 + threadIdx.x;
        if (q < cnt) {
            sb2[threadIdx.x] = w.ob2[base + q];
            se[threadIdx.x] = w.oe[base + q];
            sarg[threadIdx.x] = w.oarg[base + q];
        }
        __syncthreads();
        const int n = min(KR_BLOCK, cnt - c0);
        if (live) {
            for (int x = 0; x < n; ++x) {
                const int64_t src = b - sb2[x];
                if (src >= 0 && src < Lprev) {
                    const double v = Fprev[src] + se[x];
                    if (v < best) {
                        best = v;
                        who = sarg[x];
                    }
                }
            }
        }
        __syncthreads();
    }
    if (b < a.B) {
        Fcur[b] = live ? best : INFINITY;
        a.bp[(int64_t)k * a.B + b] = live ? who : -1;
    }
}

// Bins whose value is strictly below every earlier bin; one block.
__global__ void __launch_bounds__(KR_BLOCK) staircase_kernel(ComposeArgs a)
{
    __shared__ double sm[KR_WAVES];
    __shared__ int32_t si[KR_WAVES];
    if (*a.status != KR_OK) {
        if (threadIdx.x == 0) *a.n_stair = 0;
        return;
    }
    const double delta = a.info[0], tmin_sum = a.info[1];
    double carry = INFINITY;
    int32_t n = 0;
    for (int b0 = 0; b0 < a.B; b0 += KR_BLOCK) {
        const int b = b0 + threadIdx.x;
        const double v = b < a.B ? a.F_out[b] : INFINITY;
        double tot;
        const double before = MinF64()(carry, block_exclusive(v, (double)INFINITY, MinF64(), sm, &tot));
        const int keep = v < before;
        int32_t cnt;
        const int32_t pos = block_exclusive(keep, 0, SumI32(), si, &cnt);
        if (keep) {
            a.stair_bin[n + pos] = b;
            a.stair_Tlo[n + pos] = tmin_sum + (double)b * delta;
            a.stair_E[n + pos] = v;
        }
        n += cnt;
        carry = MinF64()(carry, tot);
    }
    if (threadIdx.x == 0) *a.n_stair = n;
}

hipError_t launch_compose(const ComposeArgs &a, const ComposeWs &w, hipEvent_t *minplus_ev,
                          hipStream_t st)
{
    hipLaunchKernelGGL(compose_init_kernel, dim3(1), dim3(64), 0, st, a);
    hipLaunchKernelGGL(compose_range_kernel, dim3(a.P), dim3(KR_BLOCK), 0, st, a, w);
    hipLaunchKernelGGL(compose_setup_kernel, dim3(1), dim3(64), 0, st, a, w);
    hipLaunchKernelGGL(compose_bin_kernel, dim3(a.P), dim3(KR_BLOCK), 0, st, a, w);
    const dim3 grid((a.B + KR_BLOCK - 1) / KR_BLOCK);
    double *buf[2] = {w.F0, w.F1};
    double *prev = a.P == 1 ? a.F_out : buf[0];
    hipLaunchKernelGGL(compose_first_kernel, grid, dim3(KR_BLOCK), 0, st, a, w, prev);
    if (minplus_ev) (void)hipEventRecord(minplus_ev[0], st);
    for (int k = 1; k < a.P; ++k) {
        double *cur = (k == a.P - 1) ? a.F_out : buf[k % 2];
        hipLaunchKernelGGL(minplus_step_kernel, grid, dim3(KR_BLOCK), 0, st, a, w, k,
                           (const double *)prev, cur);
        prev = cur;
    }
    if (minplus_ev) (void)hipEventRecord(minplus_ev[1], st);
    hipLaunchKernelGGL(staircase_kernel, dim3(1), dim3(KR_BLOCK), 0, st, a);
    return hipGetLastError();
}

// Walk the back-pointers of each query bin from the last partition to the first.
__global__ void extract_kernel(ExtractArgs a)
{
    const int q = blockIdx.x * KR_BLOCK + threadIdx.x;
    if (q >= a.n_q) return;
    int32_t *choice = a.choice + (int64_t)q * a.P;
    int64_t b = a.bins[q];
    bool ok = b >= 0 && b < a.B;
    for (int k = a.P - 1; k >= 0 && ok; --k) {
        const int32_t j = a.bp[(int64_t)k * a.B + b];
        if (j < 0) {
            ok = false;
            break;
        }
        choice[k] = j;
        b -= a.pt_bin[a.off[k] + j];
        if (b < 0) ok = false;
    }
    ok = ok && b == 0;
    double Ts = 0.0, Es = 0.0;
    if (ok) {
        for (int k = 0; k < a.P; ++k) {
            const int64_t x = a.off[k] + choice[k];
            Ts = Ts + a.T[x];
            Es = Es + a.E[x];
            if (a.cand_idx) a.choice_cand[(int64_t)q * a.P + k] = a.cand_idx[x];
        }
    } else {
        for (int k = 0; k < a.P; ++k) {
            choice[k] = -1;
            if (a.cand_idx) a.choice_cand[(int64_t)q * a.P + k] = -1;
        }
        Ts = Es = NAN;
    }
    a.T_out[q] = Ts;
    a.E_out[q] = Es;
    a.ok[q] = ok;
}

hipError_t launch_extract(const ExtractArgs &a, hipStream_t st)
{
    if (a.n_q == 0) return hipSuccess;
    hipLaunchKernelGGL(extract_kernel, dim3((a.n_q + KR_BLOCK - 1) / KR_BLOCK), dim3(KR_BLOCK), 0,
                       st, a);
    return hipGetLastError();
}

}  // namespace kr
