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

#define KR_MP_W 256     // output bins per tile
#define KR_MP_Q 4       // quarters of a partition's records per tile (block = W * Q threads)
#define KR_MP_HCAP 1024 // largest partition offset range staged in LDS

__device__ __forceinline__ double load_l2(const double *p)
{
    return bitsd(__hip_atomic_load((const uint64_t *)p, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT));
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

// Bin width, per-partition bin counts and running bin totals.  The two floating-point
// sums run sequentially in partition order on one thread, so delta and tmin_sum are
// reproducible bit for bit; the integer counts and their running totals are block
// reductions and scans (exact).
__global__ void __launch_bounds__(KR_BLOCK) compose_setup_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ double s_delta, s_tsum;
    __shared__ int64_t sc[KR_WAVES];
    if (*a.status != KR_OK) return;
    const int P = a.P, B = a.B;
    if (threadIdx.x == 0) {
        double R = 0.0, tmin_sum = 0.0;
        for (int k = 0; k < P; ++k) R = R + w.range[k];
        for (int k = 0; k < P; ++k) tmin_sum = tmin_sum + w.tmin[k];
        s_delta = a.delta_in > 0.0 ? a.delta_in : (R > 0.0 ? R / (double)(B - 1) : 1.0);
        s_tsum = tmin_sum;
    }
    __syncthreads();
    double delta = s_delta;
    for (int iter = 0;; ++iter) {
        int64_t part = 0;
        for (int k = threadIdx.x; k < P; k += KR_BLOCK) {
            const double x = floor(w.range[k] / delta);
            const int64_t m = x < (double)B ? (int64_t)x : (int64_t)B;
            w.Mk[k] = m;
            part += m;
        }
        int64_t total;
        block_exclusive(part, (int64_t)0, SumI64(), sc, &total);
        if (total + 1 <= B) break;
        if (a.delta_in > 0.0 || iter > 4096) {
            if (threadIdx.x == 0) *a.status = KR_ECAPACITY;
            return;
        }
        delta = __longlong_as_double(__double_as_longlong(delta) + 1);  // next double up
    }
    __syncthreads();
    int64_t carry = 0;  // sum of M over earlier chunks
    for (int k0 = 0; k0 < P; k0 += KR_BLOCK) {
        const int k = k0 + threadIdx.x;
        const int64_t m = k < P ? w.Mk[k] : 0;
        int64_t tot;
        const int64_t ex = block_exclusive(m, (int64_t)0, SumI64(), sc, &tot);
        if (k < P) {
            w.Lk[k] = 1 + carry + ex + m;  // 1 + sum_{j<=k} M_j
            w.eoff[k] = carry + ex + k;    // sum_{j<k} (M_j + 1)
        }
        carry += tot;
    }
    if (threadIdx.x == 0) {
        w.eoff[P] = carry + P;
        a.info[0] = delta;
        a.info[1] = s_tsum;
        *a.L_out = (int32_t)(1 + carry);
    }
}

// Offsets of every point, least energy per offset, and the list of occupied offsets,
// for one partition; eb/ea are the least-energy bits and point per offset (LDS when
// the partition's offsets fit, else global memory).
#define KR_BIN_CAP 2048
template <typename EB, typename EA>
__device__ __forceinline__ void bin_partition(const ComposeArgs &a, const ComposeWs &w, int k,
                                              EB *eb, EA *ea, int32_t *sc)
{
    const int64_t lo = a.off[k], hi = a.off[k + 1];
    const int64_t M = w.Mk[k], eo = w.eoff[k];
    const double tmin = w.tmin[k], delta = a.info[0];
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
        if (dbits(a.E[j]) == load_l2((const uint64_t *)&eb[o])) atomicMin((int32_t *)&ea[o], (int32_t)(j - lo));
    }
    __syncthreads();
    int32_t carry = 0;
    for (int64_t b0 = 0; b0 <= M; b0 += KR_BLOCK) {
        const int64_t b = b0 + threadIdx.x;
        const int32_t arg = b <= M ? load_l2((const int32_t *)&ea[b]) : 0x7FFFFFFF;
        const uint64_t ebits = b <= M ? load_l2((const uint64_t *)&eb[b]) : KR_INF_BITS;
        if (b <= M) {  // e_k of partition 0 is read back by the first step
            w.ebits[eo + b] = ebits;
            w.earg[eo + b] = arg;
        }
        const int has = arg != 0x7FFFFFFF;
        int32_t tot;
        const int32_t pos = block_exclusive(has, 0, SumI32(), sc, &tot);
        if (has) {
            w.ob2[eo + carry + pos] = (int32_t)b;
            w.oe[eo + carry + pos] = bitsd(ebits);
            w.oarg[eo + carry + pos] = arg;
        }
        carry += tot;
    }
    if (threadIdx.x == 0) w.occ[k] = carry;
}

__global__ void __launch_bounds__(KR_BLOCK) compose_bin_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ uint64_t seb[KR_BIN_CAP];
    __shared__ int32_t sea[KR_BIN_CAP];
    __shared__ int32_t sc[KR_WAVES];
    if (*a.status != KR_OK) return;
    const int k = blockIdx.x;
    if (w.Mk[k] < KR_BIN_CAP)
        bin_partition(a, w, k, seb, sea, sc);
    else
        bin_partition(a, w, k, w.ebits + w.eoff[k], w.earg + w.eoff[k], sc);
}

// F_1 and the first row of back-pointers.
__global__ void compose_first_kernel(ComposeArgs a, ComposeWs w, double *F)
{
    const int64_t b = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x;
    if (*a.status != KR_OK) return;
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

// One min-plus step on a tile of KR_MP_W output bins, for offsets up to KR_MP_HCAP:
// the window F_{k-1}[b0 - M_k, b0 + KR_MP_W) and partition k's occupied records are
// staged in LDS; the KR_MP_Q quarters of the block each take a contiguous (so
// ascending in b2) quarter of the records, and the partial minima are combined in
// quarter order with strict comparisons, so ties still go to the smallest b2.

struct MinplusLds {
    double win[KR_MP_W + KR_MP_HCAP];
    double e[KR_MP_HCAP + 1];
    int32_t off8[KR_MP_HCAP + 1];  // b2 * 8: byte offset into the window
    int32_t arg[KR_MP_HCAP + 1];
    double pbest[KR_MP_Q][KR_MP_W];
    int32_t pwho[KR_MP_Q][KR_MP_W];
};

__global__ void __launch_bounds__(KR_MP_W *KR_MP_Q)
minplus_tile_kernel(ComposeArgs a, ComposeWs w, int k, const double *Fprev, double *Fcur)
{
    __shared__ MinplusLds sm;
    if (*a.status != KR_OK) return;
    const int tid = threadIdx.x, t = tid % KR_MP_W, qtr = tid / KR_MP_W;
    const int64_t b0 = (int64_t)blockIdx.x * KR_MP_W;
    const int64_t Lprev = w.Lk[k - 1], Lcur = w.Lk[k];
    const int64_t M = w.Mk[k];
    const int cnt = w.occ[k];
    const int64_t base = w.eoff[k];
    double best = INFINITY;
    int32_t who = -1;
    if (M > KR_MP_HCAP) {
        // offsets beyond the window: every quarter-0 thread walks all records itself
        if (qtr == 0 && b0 + t < Lcur) {
            const int64_t b = b0 + t;
            for (int x = 0; x < cnt; ++x) {
                const int64_t src = b - w.ob2[base + x];
                if (src >= 0 && src < Lprev) {
                    const double v = Fprev[src] + w.oe[base + x];
                    if (v < best) {
                        best = v;
                        who = w.oarg[base + x];
                    }
                }
            }
        }
    } else {
        for (int i = tid; i < KR_MP_W + M; i += KR_MP_W * KR_MP_Q) {
            const int64_t src = b0 - M + i;
            sm.win[i] = src >= 0 && src < Lprev ? Fprev[src] : INFINITY;
        }
        for (int i = tid; i < cnt; i += KR_MP_W * KR_MP_Q) {
            sm.e[i] = w.oe[base + i];
            sm.off8[i] = w.ob2[base + i] * 8;
            sm.arg[i] = w.oarg[base + i];
        }
        __syncthreads();
        const int x0 = cnt * qtr / KR_MP_Q, x1 = cnt * (qtr + 1) / KR_MP_Q;
        const char *wl = (const char *)(sm.win + t + M);  // window entry of bin b0 + t
        int bx = -1;
#pragma unroll 4
        for (int x = x0; x < x1; ++x) {
            const double v = *(const double *)(wl - sm.off8[x]) + sm.e[x];
            bx = v < best ? x : bx;
            best = v < best ? v : best;
        }
        sm.pbest[qtr][t] = best;
        sm.pwho[qtr][t] = bx >= 0 ? sm.arg[bx] : -1;
        __syncthreads();
        if (qtr == 0) {
            who = sm.pwho[0][t];
#pragma unroll
            for (int q = 1; q < KR_MP_Q; ++q) {
                const double v = sm.pbest[q][t];
                if (v < best) {
                    best = v;
                    who = sm.pwho[q][t];
                }
            }
        }
    }
    const int64_t b = b0 + t;
    if (qtr == 0 && b < a.B) {
        const bool live = b < Lcur;
        Fcur[b] = live ? best : INFINITY;
        a.bp[(int64_t)k * a.B + b] = live ? who : -1;
    }
}

// All min-plus steps in one launch, as a wavefront over (tile, step).  Block g owns
// the KR_MP_W bins of tile g for every step: F_k of its own bins stays in LDS from one
// step to the next, and the halo F_{k-1}[b0 - M_k, b0) comes from the tiles on its
// left, which publish every step's values to the step history Fh[k][b] and then
// raise done[tile] = k.  Tile g can run step k as soon as those tiles have finished
// step k - 1, so the tiles advance as a diagonal front: a step costs one tile's
// compute, and the latency of a hand-over is paid once per tile, not once per step.
// The grid is launched cooperatively (every block resident), so a wait always ends;
// a wait that still exceeds KR_WF_POLLS polls marks the result invalid and releases
// the blocks waiting on this one.
//
// Hand-over: values and flags are written and read with device-scope relaxed atomic
// accesses, which are coherent across the chip without cache maintenance; a block
// waits for its value stores to complete before it raises its flag, and reads the
// values only after it has seen the flag.
#define KR_WF_POLLS (1 << 22)

__device__ __forceinline__ void store_dev(double *p, double v)
{
    __hip_atomic_store((uint64_t *)p, dbits(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_dev(int32_t *p, int32_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

struct WavefrontLds {
    double win[KR_MP_W + KR_MP_HCAP];  // F_{k-1}[b0 - M_k, b0 + KR_MP_W)
    double cur[KR_MP_W];               // F of the tile's own bins, last finished step
    double e[KR_MP_HCAP + 1];
    int32_t off8[KR_MP_HCAP + 1];  // b2 * 8: byte offset into the window
    int32_t arg[KR_MP_HCAP + 1];
    double pbest[KR_MP_Q][KR_MP_W];
    int32_t pwho[KR_MP_Q][KR_MP_W];
    int32_t bad;  // a wait gave up
};

__global__ void wavefront_init_kernel(int32_t *done, int G)
{
    const int g = blockIdx.x * blockDim.x + threadIdx.x;
    if (g < G) done[g] = -1;
}

__global__ void __launch_bounds__(KR_MP_W *KR_MP_Q) minplus_wavefront_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ WavefrontLds sm;
    if (*a.status != KR_OK) return;  // the same for every block
    const int tid = threadIdx.x, t = tid % KR_MP_W, qtr = tid / KR_MP_W;
    const int g = blockIdx.x;
    const int P = a.P, B = a.B;
    const int64_t b0 = (int64_t)g * KR_MP_W, b = b0 + t;
    double *const Fh = w.Fh;
    int32_t *const done = w.done;
    if (tid == 0) sm.bad = 0;

    // Waits until tiles [lo, g) have finished step k; false if a wait gave up.
    auto wait_left = [&](int lo, int k) {
        if (tid == 0) {
            for (int tt = lo; tt < g && !sm.bad; ++tt) {
                int polls = 0;
                while (load_l2(done + tt) < k) {
                    if (++polls > KR_WF_POLLS) {
                        sm.bad = 1;
                        break;
                    }
                }
            }
        }
        __syncthreads();
        return !sm.bad;
    };
    // Every thread's value stores are complete before the flag goes up.
    auto publish = [&](int k) {
        __atomic_signal_fence(__ATOMIC_SEQ_CST);  // the stores stay before the wait
        __builtin_amdgcn_s_waitcnt(0x0F70);       // vmcnt(0)
        __syncthreads();
        if (tid == 0) store_dev(done + g, k);
    };

    // step 0: F_1 = e_1
    if (qtr == 0) {
        double v = INFINITY;
        int32_t who = -1;
        if (b < B && b <= w.Mk[0]) {
            const int32_t arg = w.earg[b];
            if (arg != 0x7FFFFFFF) {
                v = bitsd(w.ebits[b]);
                who = arg;
            }
        }
        sm.cur[t] = v;
        if (b < B) {
            a.bp[b] = who;
            if (P == 1) a.F_out[b] = v;
            else store_dev(Fh + b, v);
        }
    }
    publish(0);

    for (int k = 1; k < P; ++k) {
        const int64_t Lprev = w.Lk[k - 1], Lcur = w.Lk[k];
        const int64_t M = w.Mk[k];
        const int cnt = w.occ[k];
        const int64_t base = w.eoff[k];
        const bool last = k == P - 1;
        double best = INFINITY;
        int32_t who = -1;
        if (b0 < Lcur) {
            const int lo = (int)(max((int64_t)0, b0 - M) / KR_MP_W);
            if (!wait_left(lo, k - 1)) break;
            const double *Fp = Fh + (int64_t)(k - 1) * B;
            if (M <= KR_MP_HCAP) {
                for (int i = tid; i < M; i += KR_MP_W * KR_MP_Q) {
                    const int64_t src = b0 - M + i;
                    sm.win[i] = src >= 0 && src < Lprev ? load_l2(Fp + src) : INFINITY;
                }
                for (int i = tid; i < KR_MP_W; i += KR_MP_W * KR_MP_Q) sm.win[M + i] = sm.cur[i];
                for (int i = tid; i < cnt; i += KR_MP_W * KR_MP_Q) {
                    sm.e[i] = w.oe[base + i];
                    sm.off8[i] = w.ob2[base + i] * 8;
                    sm.arg[i] = w.oarg[base + i];
                }
                __syncthreads();
                const int x0 = cnt * qtr / KR_MP_Q, x1 = cnt * (qtr + 1) / KR_MP_Q;
                const char *wl = (const char *)(sm.win + t + M);  // window entry of bin b
                int bx = -1;
#pragma unroll 4
                for (int x = x0; x < x1; ++x) {
                    const double v = *(const double *)(wl - sm.off8[x]) + sm.e[x];
                    bx = v < best ? x : bx;
                    best = v < best ? v : best;
                }
                sm.pbest[qtr][t] = best;
                sm.pwho[qtr][t] = bx >= 0 ? sm.arg[bx] : -1;
                __syncthreads();
                if (qtr == 0) {
                    who = sm.pwho[0][t];
#pragma unroll
                    for (int q = 1; q < KR_MP_Q; ++q) {
                        const double v = sm.pbest[q][t];
                        if (v < best) {
                            best = v;
                            who = sm.pwho[q][t];
                        }
                    }
                }
            } else if (qtr == 0) {
                // offsets beyond the window: each bin walks the records itself, reading
                // its own tile's F from LDS and the rest from the step history
                for (int x = 0; x < cnt; ++x) {
                    const int64_t src = b - w.ob2[base + x];
                    if (src >= 0 && src < Lprev) {
                        const double f = src >= b0 ? sm.cur[src - b0] : load_l2(Fp + src);
                        const double v = f + w.oe[base + x];
                        if (v < best) {
                            best = v;
                            who = w.oarg[base + x];
                        }
                    }
                }
            }
        }
        __syncthreads();  // every read of cur and of the window is done
        if (qtr == 0) {
            const bool live = b < Lcur;
            const double v = live ? best : INFINITY;
            sm.cur[t] = v;
            if (b < B) {
                a.bp[(int64_t)k * B + b] = live ? who : -1;
                if (last) a.F_out[b] = v;
                else if (b0 < Lcur) store_dev(Fh + (int64_t)k * B + b, v);
            }
        }
        publish(k);
    }
    if (sm.bad && tid == 0) {
        *a.status = KR_EHIP;
        store_dev(done + g, P);  // release whoever waits on this tile
    }
}

// Exclusive scan over a block of NT threads (NT / 64 waves); *total gets the aggregate.
// Every thread must call.  lds holds NT / 64 values.
template <int NT, typename T, typename Op>
__device__ __forceinline__ T block_scan_excl(T v, T identity, Op op, T *lds, T *total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const T inc = wave_inclusive(v, op);
    if (lane == 63) lds[wave] = inc;
    __syncthreads();
    T before = identity, all = identity;
#pragma unroll
    for (int q = 0; q < NT / 64; ++q) {
        const T x = lds[q];
        if (q < wave) before = op(before, x);
        all = op(all, x);
    }
    T ex = shfl_up(inc, 1);
    if (lane == 0) ex = identity;
    __syncthreads();
    *total = all;
    return op(before, ex);
}

// Bins whose value is strictly below every earlier bin.  One block: thread t takes a
// contiguous chunk of bins; a scan of the chunk minima gives each chunk the least value
// before it, a scan of the keep counts gives the output positions.
#define KR_ST_NT 1024
__global__ void __launch_bounds__(KR_ST_NT) staircase_kernel(ComposeArgs a)
{
    __shared__ double sm[KR_ST_NT / 64];
    __shared__ int32_t si[KR_ST_NT / 64];
    if (*a.status != KR_OK) {
        if (threadIdx.x == 0) *a.n_stair = 0;
        return;
    }
    const double delta = a.info[0], tmin_sum = a.info[1];
    const int C = (a.B + KR_ST_NT - 1) / KR_ST_NT;
    const int b0 = min(a.B, (int)threadIdx.x * C), b1 = min(a.B, b0 + C);
    double cmin = INFINITY;
    for (int b = b0; b < b1; ++b) cmin = MinF64()(cmin, a.F_out[b]);
    double tot;
    double run = block_scan_excl<KR_ST_NT>(cmin, (double)INFINITY, MinF64(), sm, &tot);
    const double run0 = run;
    int32_t nk = 0;
    for (int b = b0; b < b1; ++b) {
        const double v = a.F_out[b];
        if (v < run) {
            ++nk;
            run = v;
        }
    }
    int32_t n;
    int32_t pos = block_scan_excl<KR_ST_NT>(nk, 0, SumI32(), si, &n);
    run = run0;
    for (int b = b0; b < b1; ++b) {
        const double v = a.F_out[b];
        if (v < run) {
            a.stair_bin[pos] = b;
            a.stair_Tlo[pos] = tmin_sum + (double)b * delta;
            a.stair_E[pos] = v;
            ++pos;
            run = v;
        }
    }
    if (threadIdx.x == 0) *a.n_stair = n;
}

// Whether G wavefront blocks can all be resident at once on the current device (a
// cooperative launch needs it); asked once per device.
static bool wavefront_fits(int G)
{
    static int cap[64];
    static bool known[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return false;
    if (!known[dev]) {
        int coop = 0, cus = 0, per_cu = 0;
        cap[dev] = 0;
        if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) == hipSuccess &&
            coop &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
            hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &per_cu, (const void *)minplus_wavefront_kernel, KR_MP_W * KR_MP_Q, 0) == hipSuccess)
            cap[dev] = per_cu * cus;
        known[dev] = true;
    }
    return G <= cap[dev];
}

hipError_t launch_compose(const ComposeArgs &a, const ComposeWs &w, hipEvent_t *minplus_ev,
                          hipStream_t st)
{
    hipLaunchKernelGGL(compose_init_kernel, dim3(1), dim3(64), 0, st, a);
    hipLaunchKernelGGL(compose_range_kernel, dim3(a.P), dim3(KR_BLOCK), 0, st, a, w);
    hipLaunchKernelGGL(compose_setup_kernel, dim3(1), dim3(KR_BLOCK), 0, st, a, w);
    hipLaunchKernelGGL(compose_bin_kernel, dim3(a.P), dim3(KR_BLOCK), 0, st, a, w);
    const int G = (a.B + KR_MP_W - 1) / KR_MP_W;
    if (w.Fh && wavefront_fits(G)) {
        hipLaunchKernelGGL(wavefront_init_kernel, dim3((G + KR_BLOCK - 1) / KR_BLOCK),
                           dim3(KR_BLOCK), 0, st, w.done, G);
        if (minplus_ev) (void)hipEventRecord(minplus_ev[0], st);
        void *args[] = {(void *)&a, (void *)&w};
        const hipError_t e = hipLaunchCooperativeKernel((const void *)minplus_wavefront_kernel,
                                                        dim3(G), dim3(KR_MP_W * KR_MP_Q), args,
                                                        0, st);
        if (e != hipSuccess) return e;
        if (minplus_ev) (void)hipEventRecord(minplus_ev[1], st);
    } else {
        const dim3 grid((a.B + KR_BLOCK - 1) / KR_BLOCK);
        double *buf[2] = {w.F0, w.F1};
        double *prev = a.P == 1 ? a.F_out : buf[0];
        hipLaunchKernelGGL(compose_first_kernel, grid, dim3(KR_BLOCK), 0, st, a, w, prev);
        if (minplus_ev) (void)hipEventRecord(minplus_ev[0], st);
        for (int k = 1; k < a.P; ++k) {
            double *cur = (k == a.P - 1) ? a.F_out : buf[k % 2];
            hipLaunchKernelGGL(minplus_tile_kernel, dim3(G), dim3(KR_MP_W * KR_MP_Q), 0, st, a, w,
                               k, (const double *)prev, cur);
            prev = cur;
        }
        if (minplus_ev) (void)hipEventRecord(minplus_ev[1], st);
    }
    hipLaunchKernelGGL(staircase_kernel, dim3(1), dim3(KR_ST_NT), 0, st, a);
    return hipGetLastError();
}

// Walk the back-pointers of each query bin from the last partition to the first; one
// wave per query.  A step needs the chosen point's offset (a load that depends on the
// back-pointer) and then the next back-pointer (a load that depends on the offset).  The
// wave loads the next row's back-pointers for the KR_EX_SPEC bins just below the current
// one while the offset is in flight, so a step costs one memory latency when the offset
// is below KR_EX_SPEC (else one more load).
#define KR_EX_SPEC 128
__global__ void __launch_bounds__(64) extract_kernel(ExtractArgs a)
{
    const int q = blockIdx.x, lane = threadIdx.x;
    int32_t *choice = a.choice + (int64_t)q * a.P;
    int64_t b = a.bins[q];
    bool ok = b >= 0 && b < a.B;
    int32_t j = ok ? a.bp[(int64_t)(a.P - 1) * a.B + b] : -1;
    for (int k = a.P - 1; k >= 0 && ok; --k) {
        const int64_t lo = a.off[k], n = a.off[k + 1] - lo;
        if (j < 0 || j >= n) {
            ok = false;
            break;
        }
        const int32_t *row = a.bp + (int64_t)(k - 1) * a.B;
        int32_t spec[KR_EX_SPEC / 64];  // spec[i] = bp[k - 1][b - (lane + 64 i)]
#pragma unroll
        for (int i = 0; i < KR_EX_SPEC / 64; ++i) {
            const int64_t src = b - (lane + 64 * i);
            spec[i] = k > 0 && src >= 0 ? row[src] : -1;
        }
        const int64_t b2 = a.pt_bin[lo + j];
        if (lane == 0) choice[k] = j;
        b -= b2;
        if (b < 0) {
            ok = false;
            break;
        }
        if (k == 0) break;
        if (b2 < KR_EX_SPEC) {
            int32_t v = spec[0];
#pragma unroll
            for (int i = 1; i < KR_EX_SPEC / 64; ++i) v = (int)b2 / 64 == i ? spec[i] : v;
            j = __builtin_amdgcn_readlane(v, (int)b2 % 64);
        } else {
            j = row[b];
        }
    }
    ok = ok && b == 0;
    if (lane != 0) return;
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
    hipLaunchKernelGGL(extract_kernel, dim3(a.n_q), dim3(64), 0, st, a);
    return hipGetLastError();
}

}  // namespace kr
