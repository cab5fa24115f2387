// Microbatch frontier (Section 4.4, Algorithm 2 with one GPU frequency per microbatch and
// one shared configuration per partition type).  One block per frequency composes its
// scaled type frontiers with the frontier composition's rules, walks every
// non-dominated bin back to its configuration and sums it exactly in execution order;
// the union over frequencies then goes to GetFrontier.  All frequencies take one launch.
#include "kr_launch.h"
#include "kr_device.h"

namespace kr {

#define KR_MB_WIN 4096  // offsets binned on chip per pass

struct MbMinF64 {
    __device__ __forceinline__ double operator()(double a, double b) const { return b < a ? b : a; }
};
struct MbMaxF64 {
    __device__ __forceinline__ double operator()(double a, double b) const { return b > a ? b : a; }
};

// Offset of a scaled time on frequency f's grid: floor((t - tmin) / delta), clamped to
// [0, M] (the composition's binning rule).
__device__ __forceinline__ int64_t mb_offset(double t, double tmin, double delta, int64_t M)
{
    const double x = floor((t - tmin) / delta);
    return !(x > 0.0) ? 0 : (x < (double)M ? (int64_t)x : M);
}

// One block per frequency f: the frequency's whole composition and walk, with the rules of
// kr_compose_frontiers applied to the used types' points scaled by their repeat counts
// (type order): the time range of each type, the bin width (ranges summed in type order
// on one thread, then nudged up one ulp at a time until the bins fit), each type's least
// energy per offset (ties: smallest point index) and its occupied offsets, the min-plus
// steps (ties: smallest offset), the bins strictly below every earlier bin, and for each
// of those the walk back to its configuration, summed exactly in execution order and then
// over the components.  Slot f * B + q receives the q-th configuration, or +inf (choices
// -1) past the staircase or when the composition fails (an empty type, a non-finite or
// negative value, or bins that do not fit).
__global__ void __launch_bounds__(KR_BLOCK) mb_grid_kernel(MbArgs a, MbGridWs w)
{
    __shared__ double s_tmin[KR_MB_MAX_TYPES], s_range[KR_MB_MAX_TYPES], s_delta;
    __shared__ int64_t s_M[KR_MB_MAX_TYPES], s_L[KR_MB_MAX_TYPES];
    __shared__ int32_t s_status, s_nstair;
    __shared__ double scd[KR_WAVES];
    __shared__ int32_t sci[KR_WAVES];
    __shared__ uint64_t s_eb[KR_MB_WIN];
    __shared__ int32_t s_ea[KR_MB_WIN];
    const int f = blockIdx.x, tid = threadIdx.x, B = a.B, Ku = a.Ku;
    const size_t wb = (size_t)f * B;
    int32_t *const ob2 = w.ob2 + wb, *const oarg = w.oarg + wb;
    double *const oe = w.oe + wb;
    double *const F0 = w.F + (size_t)f * 2 * B, *const F1 = F0 + B;
    int32_t *const bp = w.bp + (size_t)f * a.K * B;
    int32_t *const stair = w.stair + (size_t)f * B;
    if (tid == 0) s_status = KR_OK;
    __syncthreads();

    // time range of each type's scaled points; their times and energies are checked
    for (int u = 0; u < Ku; ++u) {
        const int t = a.used[u];
        const int64_t lo = a.seg_off[t * a.F + f], n = a.seg_off[t * a.F + f + 1] - lo;
        const double m = (double)a.count[u];
        double mn = INFINITY, mx = -INFINITY;
        bool bad = false;
        for (int64_t j = tid; j < n; j += KR_BLOCK) {
            const double ts = m * a.T[lo + j], es = m * a.E[lo + j];
            mn = ts < mn ? ts : mn;
            mx = ts > mx ? ts : mx;
            bad = bad || !(dbits(fabs(ts)) < KR_INF_BITS) || !(dbits(es + 0.0) < KR_INF_BITS);
        }
        if (__ballot(bad) && (tid & 63) == 0) s_status = KR_ENONFINITE;
        mn = block_reduce(mn, (double)INFINITY, MbMinF64(), scd);
        mx = block_reduce(mx, -(double)INFINITY, MbMaxF64(), scd);
        if (tid == 0) {
            if (n <= 0) s_status = KR_EINVAL;
            s_tmin[u] = mn;
            s_range[u] = mx - mn;
        }
    }
    __syncthreads();
    // bin width and the types' offset ranges M and reachable bins L
    if (tid == 0 && s_status == KR_OK) {
        double R = 0.0;
        for (int u = 0; u < Ku; ++u) R = R + s_range[u];
        double delta = R > 0.0 ? R / (double)(B - 1) : 1.0;
        for (int iter = 0;; ++iter) {
            int64_t tot = 0;
            for (int u = 0; u < Ku; ++u) {
                const double x = floor(s_range[u] / delta);
                const int64_t mm = x < (double)B ? (int64_t)x : (int64_t)B;
                s_M[u] = mm;
                tot += mm;
            }
            if (tot + 1 <= B) break;
            if (iter > 4096) {
                s_status = KR_ECAPACITY;
                break;
            }
            delta = __longlong_as_double(__double_as_longlong(delta) + 1);  // next double up
        }
        int64_t L = 1;
        for (int u = 0; u < Ku; ++u) {
            L += s_M[u];
            s_L[u] = L;
        }
        s_delta = delta;
    }
    __syncthreads();
    const bool good = s_status == KR_OK;
    const double delta = s_delta;

    if (good) {
        for (int u = 0; u < Ku; ++u) {
            const int t = a.used[u];
            const int64_t lo = a.seg_off[t * a.F + f], n = a.seg_off[t * a.F + f + 1] - lo;
            const double m = (double)a.count[u], tmin = s_tmin[u];
            const int64_t M = s_M[u];
            // least energy per offset, then the smallest point index that has it, on
            // chip for a window of KR_MB_WIN offsets at a time; the occupied offsets
            // go to the block's list in ascending order
            int32_t occ = 0;
            for (int64_t c0 = 0; c0 <= M; c0 += KR_MB_WIN) {
                const int cn = (int)min((int64_t)KR_MB_WIN, M + 1 - c0);
                for (int b = tid; b < cn; b += KR_BLOCK) {
                    s_eb[b] = KR_INF_BITS;
                    s_ea[b] = 0x7FFFFFFF;
                }
                __syncthreads();
                for (int64_t j = tid; j < n; j += KR_BLOCK) {
                    const int64_t o = mb_offset(m * a.T[lo + j], tmin, delta, M) - c0;
                    if (o >= 0 && o < cn)
                        atomicMin((unsigned long long *)&s_eb[o],
                                  (unsigned long long)dbits(m * a.E[lo + j] + 0.0));
                }
                __syncthreads();
                for (int64_t j = tid; j < n; j += KR_BLOCK) {
                    const int64_t o = mb_offset(m * a.T[lo + j], tmin, delta, M) - c0;
                    if (o >= 0 && o < cn && dbits(m * a.E[lo + j] + 0.0) == s_eb[o])
                        atomicMin(&s_ea[o], (int32_t)j);
                }
                __syncthreads();
                for (int b0 = 0; b0 < cn; b0 += KR_BLOCK) {
                    const int b = b0 + tid;
                    const int32_t arg = b < cn ? s_ea[b] : 0x7FFFFFFF;
                    const int has = arg != 0x7FFFFFFF;
                    int32_t tot;
                    const int32_t pos = block_exclusive(has, 0, SumI32(), sci, &tot);
                    if (has) {
                        ob2[occ + pos] = (int32_t)(c0 + b);
                        oe[occ + pos] = bitsd(s_eb[b]);
                        oarg[occ + pos] = arg;
                    }
                    occ += tot;
                }
                __syncthreads();
            }
            // F_1 = e_1, then F_u[b] = min over occupied b2 of F_{u-1}[b - b2] + e_u[b2]
            double *const Fc = (u & 1) ? F1 : F0;
            const double *const Fp = (u & 1) ? F0 : F1;
            int32_t *const bpu = bp + (size_t)u * B;
            const int64_t Lu = s_L[u], Lp = u > 0 ? s_L[u - 1] : 0;
            for (int b = tid; b < B; b += KR_BLOCK) {
                double best = INFINITY;
                int32_t who = -1;
                if (u > 0 && b < Lu) {
                    for (int x = 0; x < occ; ++x) {
                        const int64_t src = b - ob2[x];
                        if (src >= 0 && src < Lp) {
                            const double v = Fp[src] + oe[x];
                            if (v < best) {
                                best = v;
                                who = oarg[x];
                            }
                        }
                    }
                }
                Fc[b] = best;
                bpu[b] = who;
            }
            __syncthreads();
            if (u == 0) {  // F_1 = e_1: the occupied offsets of the first type
                for (int x = tid; x < occ; x += KR_BLOCK) {
                    Fc[ob2[x]] = oe[x];
                    bpu[ob2[x]] = oarg[x];
                }
                __syncthreads();
            }
        }
        // bins strictly below every earlier bin of F_Ku
        const double *const Fl = ((Ku - 1) & 1) ? F1 : F0;
        double before = INFINITY;
        int32_t ns = 0;
        for (int b0 = 0; b0 < B; b0 += KR_BLOCK) {
            const int b = b0 + tid;
            const double v = b < B ? Fl[b] : INFINITY;
            // least value of the bins before b in this chunk
            const double inc = wave_inclusive(v, MbMinF64());
            double ex = shfl_up(inc, 1);
            if ((tid & 63) == 0) ex = INFINITY;
            if ((tid & 63) == 63) scd[tid >> 6] = inc;
            __syncthreads();
            double wpre = INFINITY, call = INFINITY;
#pragma unroll
            for (int q = 0; q < KR_WAVES; ++q) {
                const double x = scd[q];
                if (q < (tid >> 6)) wpre = MbMinF64()(wpre, x);
                call = MbMinF64()(call, x);
            }
            __syncthreads();
            const double run = MbMinF64()(before, MbMinF64()(wpre, ex));
            const int keep = v < run;
            int32_t tot;
            const int32_t pos = block_exclusive(keep, 0, SumI32(), sci, &tot);
            if (keep) stair[ns + pos] = b;
            ns += tot;
            before = MbMinF64()(before, call);
        }
        if (tid == 0) s_nstair = ns;
        __syncthreads();
    }

    // each staircase bin walked back to its configuration and summed exactly
    const int nst = good ? s_nstair : 0;
    for (int q = tid; q < B; q += KR_BLOCK) {
        const int64_t slot = (int64_t)f * B + q;
        int32_t *ch = a.slot_choice + slot * a.K;
        int32_t choice[KR_MB_MAX_TYPES];
        bool ok = q < nst;
        if (ok) {
            int64_t b = stair[q];
            for (int u = Ku - 1; u >= 0 && ok; --u) {
                const int32_t j = bp[(size_t)u * B + b];
                ok = j >= 0;
                choice[u] = j;
                if (ok) {
                    const int64_t lo = a.seg_off[a.used[u] * a.F + f];
                    b -= mb_offset((double)a.count[u] * a.T[lo + j], s_tmin[u], delta, s_M[u]);
                    ok = b >= 0;
                }
            }
            ok = ok && b == 0;
        }
        for (int t = 0; t < a.K; ++t) ch[t] = -1;
        if (!ok) {
            a.slot_T[slot] = INFINITY;
            a.slot_E[slot] = INFINITY;
            continue;
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
        for (int u = 0; u < Ku; ++u) ch[a.used[u]] = choice[u];
    }
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

hipError_t launch_mb_grid(const MbArgs &a, const MbGridWs &w, hipStream_t st)
{
    hipLaunchKernelGGL(mb_grid_kernel, dim3(a.F), dim3(KR_BLOCK), 0, st, a, w);
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
