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
#include "kr_wave.h"

#include <utility>

namespace kr {

struct MinF64 {
    __device__ __forceinline__ double operator()(double a, double b) const { return b < a ? b : a; }
};
struct MaxF64 {
    __device__ __forceinline__ double operator()(double a, double b) const { return b > a ? b : a; }
};
struct MaxI64 {
    __device__ __forceinline__ int64_t operator()(int64_t a, int64_t b) const { return b > a ? b : a; }
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

__device__ __forceinline__ void store_dev(uint64_t *p, uint64_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_dev(int32_t *p, int32_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void compose_init_kernel(ComposeArgs a, ComposeWs w)
{
    if (threadIdx.x == 0) {
        *a.status = KR_OK;
        *w.ticket = 0;
    }
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
    bool bad = false;  // a non-finite time, or an energy that is not a finite value >= 0
    for (int64_t j = lo + threadIdx.x; j < hi; j += KR_BLOCK) {
        const double t = a.T[j];
        mn = t < mn ? t : mn;
        mx = t > mx ? t : mx;
        bad = bad || !(dbits(fabs(t)) < KR_INF_BITS) || !(dbits(a.E[j] + 0.0) < KR_INF_BITS);
    }
    if (__ballot(bad) && (threadIdx.x & 63) == 0) store_dev(a.status, (int32_t)KR_ENONFINITE);
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
    constexpr int kChunk = 1024;
    __shared__ double s_delta, s_tsum;
    __shared__ double s_range[kChunk], s_tmin[kChunk];
    __shared__ int64_t sc[KR_WAVES];
    if (*a.status != KR_OK) return;
    const int P = a.P, B = a.B;
    // the sums in partition order, by thread 0 from LDS copies the block loads together
    double R = 0.0, tmin_sum = 0.0;
    for (int k0 = 0; k0 < P; k0 += kChunk) {
        const int n = min(kChunk, P - k0);
        for (int k = threadIdx.x; k < n; k += KR_BLOCK) {
            s_range[k] = w.range[k0 + k];
            s_tmin[k] = w.tmin[k0 + k];
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            int k = 0;
            for (; k + 8 <= n; k += 8) {
                double r8[8], t8[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    r8[q] = s_range[k + q];
                    t8[q] = s_tmin[k + q];
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    R = R + r8[q];
                    tmin_sum = tmin_sum + t8[q];
                }
            }
            for (; k < n; ++k) {
                R = R + s_range[k];
                tmin_sum = tmin_sum + s_tmin[k];
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
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
    int64_t mx = 0;     // largest M seen by this thread
    for (int k0 = 0; k0 < P; k0 += KR_BLOCK) {
        const int k = k0 + threadIdx.x;
        const int64_t m = k < P ? w.Mk[k] : 0;
        mx = m > mx ? m : mx;
        int64_t tot;
        const int64_t ex = block_exclusive(m, (int64_t)0, SumI64(), sc, &tot);
        if (k < P) {
            w.Lk[k] = 1 + carry + ex + m;  // 1 + sum_{j<=k} M_j
            w.eoff[k] = carry + ex + 8 * (int64_t)k;  // sum_{j<k} (M_j + 8)
        }
        carry += tot;
    }
    mx = block_reduce(mx, (int64_t)0, MaxI64(), sc);
    if (threadIdx.x == 0) {
        *w.mmax = mx;
        w.eoff[P] = carry + 8 * (int64_t)P;
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
        atomicMin((unsigned long long *)&eb[o], (unsigned long long)dbits(a.E[j] + 0.0));
    }
    __syncthreads();
    for (int64_t j = lo + threadIdx.x; j < hi; j += KR_BLOCK) {
        const int32_t o = a.pt_bin[j];
        if (dbits(a.E[j] + 0.0) == load_l2((const uint64_t *)&eb[o]))
            atomicMin((int32_t *)&ea[o], (int32_t)(j - lo));
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
    if (threadIdx.x < 7) {  // the table runs on to a multiple of 8 past M with empty offsets
        w.ebits[eo + M + 1 + threadIdx.x] = KR_INF_BITS;
        w.earg[eo + M + 1 + threadIdx.x] = 0x7FFFFFFF;
    }
}


// All min-plus steps in one launch, as a wavefront over (tile, step).  Block g owns
// the KR_MP_W bins of tile g for every step: F_k of its own bins stays in LDS from one
// step to the next, and the halo F_{k-1}[b0 - M_k, b0) comes from the tiles on its
// left through the step history Fh[k][b].  A tile publishes only what other tiles read:
// row k, its bins within M_{k+1} of its right edge and below L_k.  Before the launch
// those entries are set to KR_UNSET, a NaN pattern no step writes; a reader loads an
// entry until it holds something else, so every value is its own ready flag and a
// hand-over costs one store and one load.  Tile g runs step k as soon as the tiles on
// its left have finished step k - 1, so the tiles advance as a diagonal front.  The
// next step's halo and records are loaded while the current step computes.
//
// Tiles are handed out by an atomic ticket taken when a block starts, not by block
// index, so the tile a block waits on (always further left, a smaller ticket) belongs to
// a block that started earlier and is resident or finished: the waits end without any
// guarantee that the whole grid is resident at once, and without a cooperative launch.
// A wait that still exceeds KR_WF_POLLS polls sets the status to KR_EHIP, and every
// other waiter gives up as soon as it sees that status.  Entries are written and read with
// device-scope relaxed atomic accesses, which are coherent across the chip without
// cache maintenance; each is written at most once per launch, after the fill kernel.
#define KR_WF_POLLS (1 << 22)
#define KR_UNSET 0x7FF4B1A5C0DE0000ull


// Whether bin x of row k is read by another tile: within M_{k+1} of its tile's right
// edge and below L_k (M1 = M_{k+1}, L = L_k).
__device__ __forceinline__ bool exported(int64_t x, int64_t M1, int64_t L)
{
    return x < L && (x % KR_MP_W) >= KR_MP_W - M1;
}

// Blocks 0 .. P-1 bin partition k = blockIdx.x.  Blocks P .. 2P-2 mark every entry of
// step-history row k = blockIdx.x - P that some tile will publish as unwritten.  The
// two are independent (both need only the setup), so they share one launch.
__global__ void __launch_bounds__(KR_BLOCK) compose_bin_fill_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ uint64_t seb[KR_BIN_CAP];
    __shared__ int32_t sea[KR_BIN_CAP];
    __shared__ int32_t sc[KR_WAVES];
    if (*a.status != KR_OK) return;
    if ((int)blockIdx.x >= a.P) {
        const int k = blockIdx.x - a.P;
        const int64_t L = min(w.Lk[k], (int64_t)a.B), M1 = w.Mk[k + 1];
        uint64_t *row = (uint64_t *)w.Fh + (int64_t)k * a.B;
        for (int64_t x = threadIdx.x; x < L; x += KR_BLOCK)
            if (exported(x, M1, L)) row[x] = KR_UNSET;
        return;
    }
    const int k = blockIdx.x;
    if (w.Mk[k] < KR_BIN_CAP)
        bin_partition(a, w, k, seb, sea, sc);
    else
        bin_partition(a, w, k, w.ebits + w.eoff[k], w.earg + w.eoff[k], sc);
}

#define KR_WF_MC 512  // steps per chunk of the block's step-metadata ring
// Window entries below offset H (read only by padding offsets).  Odd, with an even row
// length, so that a thread's group reads (which start 7 entries below an even bin)
// begin at an even index of either row: 16-byte aligned.
#define KR_WF_LO 9
#define KR_WF_S 8     // offset slices of the dense scan (block = 128 bin pairs x 8 slices)

struct WavefrontLds {
    // Window of step k in buffer k & 1: win[LO + H + i] = F_{k-1}[b0 + i] for i in
    // [-M_k, W), the halo and then the tile's own bins (one spare entry keeps the row
    // length even).
    alignas(16) double win[2][KR_WF_LO + KR_MP_HCAP + KR_MP_W + 1];
    // Records of step k in buffer k & 1: the dense least-energy table e_k[0 .. 8
    // ceil((M_k + 1) / 8)) (INFINITY past M_k) with its points, or the occupied offsets
    // only (b2 * 8 in off8).
    double e[2][KR_MP_HCAP + 8];
    int32_t off8[2][KR_MP_HCAP + 8];
    int32_t arg[2][KR_MP_HCAP + 8];
    double pbest[KR_WF_S][KR_MP_W];  // partial minima per slice (or quarter) and bin
    int32_t pidx[KR_WF_S][KR_MP_W];  // their 8-offset group (dense) or point (sparse)
    int4 meta[2][KR_WF_MC];  // (M_k, L_k, first record, records) at [(k / MC) & 1][k % MC]
    int32_t bad;             // a wait was given up
    int32_t tile;            // this block's tile (its ticket)
};

// Whether step k scans its dense offset table (about 2.25 instructions per pair) rather
// than its occupied offsets (about 7 per pair).
__device__ __forceinline__ bool dense_step(int4 m) { return 18 * ((m.x + 8) / 8) <= 7 * m.w; }

typedef const __attribute__((address_space(4))) double const_f64;

// Roles inside a block: the first KR_MP_W threads (four waves) combine the partial
// minima and store the step's results; the other threads load the next step's records
// and halo while the step computes and move them into LDS at its end.  The two never
// mix, so a wave that stores never has to wait for its stores to complete, and a wave
// that waits for its loads has no stores in flight (one in-order counter covers both).
__global__ void __launch_bounds__(KR_MP_W *KR_MP_Q) minplus_wavefront_kernel(ComposeArgs a, ComposeWs w)
{
    constexpr int NT = KR_MP_W * KR_MP_Q, H = KR_MP_HCAP, MC = KR_WF_MC, LO = KR_WF_LO;
    constexpr int NS = NT - KR_MP_W;  // loader threads
    __shared__ WavefrontLds sm;
    if (*a.status != KR_OK) return;  // the same for every block
    const int tid = threadIdx.x, t = tid % KR_MP_W;
    const int qtr = __builtin_amdgcn_readfirstlane(tid / KR_MP_W);
    const bool loader = qtr != 0;
    const int s = tid - KR_MP_W;  // loader index
    const int P = a.P, B = a.B;
    if (tid == 0) sm.tile = atomicAdd(w.ticket, 1);
    __syncthreads();
    const int64_t b0 = (int64_t)sm.tile * KR_MP_W, b = b0 + t;
    uint64_t *const Fh = (uint64_t *)w.Fh;
    auto window = [&](int k) { return sm.win[k & 1] + LO + H; };  // window(k)[i] = F_{k-1}[b0 + i]

    auto load_meta = [&](int c) {  // chunk c of the step metadata into its ring slot
        for (int i = s; i < MC; i += NS) {
            const int k = c * MC + i;
            if (k < P)
                sm.meta[c & 1][i] = make_int4((int)w.Mk[k], (int)w.Lk[k], (int)w.eoff[k], w.occ[k]);
        }
    };
    auto meta = [&](int k) { return sm.meta[(k / MC) & 1][k % MC]; };  // x M, y L, z base, w count
    if (tid == 0) sm.bad = 0;
    for (int i = tid; i < 2 * (LO + H); i += NT)  // read by padding offsets only
        sm.win[i / (LO + H)][i % (LO + H)] = INFINITY;
    if (loader) {
        load_meta(0);
        load_meta(1);
    }
    __syncthreads();

    auto gave_up = [&]() {
        return __hip_atomic_load(&sm.bad, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) != 0;
    };
    // Value of the published entry *p, first loaded as v: loads it again until it has
    // been written.  INFINITY once waiting has been given up.
    auto fetch = [&](const uint64_t *p, uint64_t v) -> double {
        for (int polls = 1; v == KR_UNSET; ++polls) {
            if (gave_up()) return INFINITY;
            if (polls % 1024 == 0) {
                const bool over = polls > KR_WF_POLLS;
                if (over) store_dev(a.status, (int32_t)KR_EHIP);
                if (over || load_l2(a.status) != KR_OK) {
                    __hip_atomic_store(&sm.bad, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                    return INFINITY;
                }
            }
            __builtin_amdgcn_s_sleep(1);
            v = load_l2(p);
        }
        return bitsd(v);
    };

    // Loader registers: the next step's records and halo entries.  A wave issues a
    // round of loads only if some lane of it has an entry in that round (dense steps
    // skip the occupied-offset list); within such a round the loads are unconditional
    // (a lane with nothing to load reads a valid dummy address).
    uint64_t hv[2], re[2];
    int32_t ro[2], ra[2];
    auto halo_src = [&](int4 m, int Lprev, int h, int64_t &src) {
        const int i = s + h * NS;
        src = b0 - m.x + i;
        return m.x <= H && i < m.x && src >= 0 && src < Lprev;
    };
    const int ws = __builtin_amdgcn_readfirstlane(s & ~63);  // the wave's first loader index
    auto issue = [&](int k, int4 m, int Lprev) {  // loads for step k
        const bool dense = dense_step(m);
        const int n = dense ? 8 * ((m.x + 8) / 8) : m.w;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            if (ws + r * NS >= n) continue;  // wave-uniform
            const int i = s + r * NS;
            const int64_t xd = m.z + max(0, min(i, m.x + 7)), xs = m.z + max(0, min(i, m.w - 1));
            if (dense) {
                re[r] = w.ebits[xd];
                ra[r] = w.earg[xd];
            } else {
                re[r] = *(const uint64_t *)(w.oe + xs);
                ra[r] = w.oarg[xs];
                ro[r] = w.ob2[xs];
            }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (ws + h * NS >= m.x) continue;  // wave-uniform
            int64_t src;
            const bool need = halo_src(m, Lprev, h, src);
            hv[h] = load_l2(Fh + (int64_t)(k - 1) * B + (need ? src : 0));
        }
    };
    auto stage = [&](int k, int4 m, int Lprev) {  // the loads of issue(k) into LDS
        const int buf = k & 1;
        const bool dense = dense_step(m);
        const int n = dense ? 8 * ((m.x + 8) / 8) : m.w;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int i = s + r * NS;
            if (i < n) {
                sm.e[buf][i] = bitsd(re[r]);
                if (!dense) sm.off8[buf][i] = ro[r] * 8;
                sm.arg[buf][i] = ra[r];
            }
        }
        if (b0 < m.y) {
            double *const wn = window(k);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                int64_t src;
                const int i = s + h * NS;
                if (i < m.x) {
                    const bool need = halo_src(m, Lprev, h, src);
                    wn[i - m.x] = need ? fetch(Fh + (int64_t)(k - 1) * B + src, hv[h]) : INFINITY;
                }
            }
        }
        asm volatile("" ::"v"(hv[0]), "v"(hv[1]), "v"(re[0]), "v"(re[1]), "v"(ro[0]), "v"(ro[1]),
                     "v"(ra[0]), "v"(ra[1]));
    };
    // Whether this loader wave has records or halo entries of step k to move (most
    // loader waves have none when the offset range is short).
    auto busy = [&](int4 m) { return ws < max(dense_step(m) ? 8 * ((m.x + 8) / 8) : m.w, m.x); };
    auto publish = [&](int k, double v, int M1, int L) {
        uint64_t bits = dbits(v);
        if (bits == KR_UNSET) bits = 0x7FF8000000000000ull;  // keep the marker unique
        if (exported(b, M1, L)) store_dev(Fh + (int64_t)k * B + b, bits);
    };

    // step 0: F_1 = e_1, into the window of step 1
    const int4 m0 = meta(0);
    if (!loader) {
        double v = INFINITY;
        int32_t who = -1;
        if (b < B && b <= m0.x) {
            const int32_t arg = w.earg[b];
            if (arg != 0x7FFFFFFF) {
                v = bitsd(w.ebits[b]);
                who = arg;
            }
        }
        window(1)[t] = v;
        if (b < B) {
            a.bp[b] = who;
            if (a.bp_off) a.bp_off[b] = who >= 0 ? (int32_t)b : -1;  // its offset is b
            if (P == 1) a.F_out[b] = v;
            else publish(0, v, meta(1).x, m0.y);
        }
    }

    if (*w.mmax > H) {
        // Some partition's offsets do not fit the window: every combining thread walks
        // all records of its bin, reading its own tile's F from LDS and the rest from
        // the step history.  The loops of the two modes share no code.
        int4 mc = m0;
        for (int k = 1; k < P; ++k) {
            __syncthreads();  // F_{k-1} of the tile and the metadata of step k are in LDS
            const int4 mp = mc;
            mc = meta(k);
            const bool last = k == P - 1;
            const int M1 = last ? 0 : meta(k + 1).x;
            const double *const wc = window(k);
            double best = INFINITY;
            int32_t who = -1, wo = -1;  // point and its offset
            if (!loader && b0 < mc.y) {
                for (int x = 0; x < mc.w; ++x) {
                    const int64_t src = b - w.ob2[mc.z + x];
                    if (src >= 0 && src < mp.y) {
                        const uint64_t *p = Fh + (int64_t)(k - 1) * B + src;
                        const double f = src >= b0 ? wc[src - b0] : fetch(p, load_l2(p));
                        const double v = f + w.oe[mc.z + x];
                        if (v < best) {
                            best = v;
                            who = w.oarg[mc.z + x];
                            wo = w.ob2[mc.z + x];
                        }
                    }
                }
            }
            __syncthreads();  // the metadata of step k has been read
            if (!loader) {
                const bool live = b < mc.y;
                const double v = live ? best : INFINITY;
                window(k + 1)[t] = v;
                if (b < B) {
                    a.bp[(int64_t)k * B + b] = live ? who : -1;
                    if (a.bp_off) a.bp_off[(int64_t)k * B + b] = live ? wo : -1;
                    if (last) a.F_out[b] = v;
                    else publish(k, v, M1, mc.y);
                }
            } else if ((k + 1) % MC == 0) {
                load_meta((k + 1) / MC + 1);  // replaces chunk (k + 1) / MC - 1
            }
        }
        return;
    }

    if (loader && P > 1 && busy(meta(1))) {
        issue(1, meta(1), m0.y);
        stage(1, meta(1), m0.y);
    }
    // The point behind bin b0 + u's least value best of step k, and its offset: the
    // part's record (sparse) or the first offset of 8-offset group idx that reaches best
    // (dense).  (-1, -1) if none.
    auto point = [&](int k, double best, int idx, bool dense, int u, int32_t &off) -> int32_t {
        off = -1;
        if (idx < 0) return -1;
        if (!dense) {
            off = sm.off8[k & 1][idx] / 8;
            return sm.arg[k & 1][idx];
        }
        const double *const wp = window(k);
        const double *const ep = sm.e[k & 1];
        const int i8 = 8 * idx;
        int o = 7;
#pragma unroll
        for (int d = 7; d >= 0; --d) o = wp[u - i8 - d] + ep[i8 + d] == best ? d : o;
        off = i8 + o;
        return sm.arg[k & 1][i8 + o];
    };
    // Least value and its part's index for bin b0 + u from the partial minima.
    auto combine = [&](bool dense, int u, double &best, int32_t &idx) {
        double pv[KR_WF_S];
        int32_t pi[KR_WF_S];
#pragma unroll
        for (int q = 0; q < KR_WF_S; ++q) {  // all read at once; a sparse step fills KR_MP_Q
            pv[q] = sm.pbest[q][u];
            pi[q] = sm.pidx[q][u];
        }
        // the first part (in offset order) with the least value, as a tree: a later part
        // replaces an earlier one only if strictly less.  A part with no candidate holds
        // (INFINITY, -1), so with none at all the result is (INFINITY, -1).
        if (!dense) {
#pragma unroll
            for (int q = KR_MP_Q; q < KR_WF_S; ++q) {
                pv[q] = INFINITY;
                pi[q] = -1;
            }
        }
#pragma unroll
        for (int d = 1; d < KR_WF_S; d *= 2)
#pragma unroll
            for (int q = 0; q + d < KR_WF_S; q += 2 * d)
                if (pv[q + d] < pv[q]) {
                    pv[q] = pv[q + d];
                    pi[q] = pi[q + d];
                }
        best = pv[0];
        idx = pi[0];
    };
    for (int k = 1; k < P; ++k) {
        __syncthreads();  // window and records of step k are in LDS
        const int4 mc = meta(k);
        const bool last = k == P - 1;
        const bool active = b0 < mc.y;
        const bool dense = dense_step(mc);
        const int4 mn = meta(last ? k : k + 1);
        const bool moves = loader && !last && busy(mn);
        if (moves) {
            // ahead of the SIMD's other waves: the loads then fly during their scans
            __builtin_amdgcn_s_setprio(2);
            issue(k + 1, mn, mc.y);
            __builtin_amdgcn_s_setprio(0);
        }
        const int buf = k & 1;
        const double *const wc = window(k);
        if (active) {
            if (dense) {
                // Thread (pair j, slice q): bins 2j and 2j + 1 over the slice's groups of
                // 8 offsets.  A group needs 9 window entries and 8 table entries; the
                // table comes from memory through the scalar cache (it does not change
                // during the launch).  The first 8 window entries are four aligned
                // 16-byte reads: threads 16 bytes apart then read without LDS bank
                // conflicts (8-byte reads at that stride conflict four ways).  The
                // running minimum takes one v_min per pair; the group where it last fell
                // is kept and rescanned when combining.
                const int j = tid % (KR_MP_W / 2);
                const int q = __builtin_amdgcn_readfirstlane(tid / (KR_MP_W / 2));
                const int ng = (mc.x + 8) / 8;
                const int g0 = __builtin_amdgcn_readfirstlane(ng * q / KR_WF_S);
                const int g1 = __builtin_amdgcn_readfirstlane(ng * (q + 1) / KR_WF_S);
                const_f64 *et = (const_f64 *)(w.ebits + __builtin_amdgcn_readfirstlane(mc.z));
                double best0 = INFINITY, best1 = INFINITY;
                int bg0 = -1, bg1 = -1;
                // one group of 8 offsets: updates the two running minima
                auto group = [&](int g, const double *x, const double *e) {
                    double v0[8], v1[8];  // offset 8g + o for bins 2j and 2j + 1
#pragma unroll
                    for (int o = 0; o < 8; ++o) {
                        v0[o] = x[7 - o] + e[o];
                        v1[o] = x[8 - o] + e[o];
                    }
                    const double m0v = vmin(vmin(vmin(v0[0], v0[1]), vmin(v0[2], v0[3])),
                                            vmin(vmin(v0[4], v0[5]), vmin(v0[6], v0[7])));
                    const double m1v = vmin(vmin(vmin(v1[0], v1[1]), vmin(v1[2], v1[3])),
                                            vmin(vmin(v1[4], v1[5]), vmin(v1[6], v1[7])));
                    bg0 = m0v < best0 ? g : bg0;
                    bg1 = m1v < best1 ? g : bg1;
                    best0 = vmin(best0, m0v);
                    best1 = vmin(best1, m1v);
                };
                // A slice of three groups (17 to 24 groups over 8 slices) takes them in
                // one round, all loads issued together, so the slowest slice pays one
                // load latency like the others.  Otherwise two groups a round; an odd
                // last round repeats its group, which cannot lower a minimum twice.
                if (g1 - g0 == 3) {  // wave-uniform
                    const double *wa = wc + 2 * j - 8 * g0 - 7;
                    double xa[9], xb[9], xc[9], ea[8], eb[8], ec[8];
#pragma unroll
                    for (int d = 0; d < 4; ++d) {
                        const double2 va = ((const double2 *)wa)[d];
                        const double2 vb = ((const double2 *)(wa - 8))[d];
                        const double2 vc = ((const double2 *)(wa - 16))[d];
                        xa[2 * d] = va.x;
                        xa[2 * d + 1] = va.y;
                        xb[2 * d] = vb.x;
                        xb[2 * d + 1] = vb.y;
                        xc[2 * d] = vc.x;
                        xc[2 * d + 1] = vc.y;
                    }
                    xa[8] = wa[8];
                    xb[8] = wa[0];
                    xc[8] = wa[-8];
#pragma unroll
                    for (int o = 0; o < 8; ++o) {
                        ea[o] = et[8 * g0 + o];
                        eb[o] = et[8 * g0 + 8 + o];
                        ec[o] = et[8 * g0 + 16 + o];
                    }
                    group(g0, xa, ea);
                    group(g0 + 1, xb, eb);
                    group(g0 + 2, xc, ec);
                } else
                for (int g = g0; g < g1; g += 2) {
                    const int h = min(g + 1, g1 - 1);
                    const double *wa = wc + 2 * j - 8 * g - 7, *wb = wc + 2 * j - 8 * h - 7;
                    double xa[9], xb[9], ea[8], eb[8];  // xa[d]: F at bin 2j + d - 7 - 8g
#pragma unroll
                    for (int d = 0; d < 4; ++d) {
                        const double2 va = ((const double2 *)wa)[d];
                        const double2 vb = ((const double2 *)wb)[d];
                        xa[2 * d] = va.x;
                        xa[2 * d + 1] = va.y;
                        xb[2 * d] = vb.x;
                        xb[2 * d + 1] = vb.y;
                    }
                    xa[8] = wa[8];
                    xb[8] = wb[8];
#pragma unroll
                    for (int o = 0; o < 8; ++o) {
                        ea[o] = et[8 * g + o];
                        eb[o] = et[8 * h + o];
                    }
                    group(g, xa, ea);
                    group(h, xb, eb);
                }
                sm.pbest[q][2 * j] = best0;
                sm.pbest[q][2 * j + 1] = best1;
                sm.pidx[q][2 * j] = bg0;
                sm.pidx[q][2 * j + 1] = bg1;
            } else {
                const int x0 = mc.w * qtr / KR_MP_Q, x1 = mc.w * (qtr + 1) / KR_MP_Q;
                const char *wl = (const char *)(wc + t);
                double best = INFINITY;
                int bx = -1;
#pragma unroll 4
                for (int x = x0; x < x1; ++x) {
                    const double v = *(const double *)(wl - sm.off8[buf][x]) + sm.e[buf][x];
                    bx = v < best ? x : bx;
                    best = v < best ? v : best;
                }
                sm.pbest[qtr][t] = best;
                sm.pidx[qtr][t] = bx;  // the record; its point and offset are read at the end
            }
        }
        __syncthreads();  // every partial minimum is in LDS
        if (!loader) {
            double best = INFINITY;
            int32_t idx = -1;
            if (active) combine(dense, t, best, idx);
            const bool live = b < mc.y;
            const double v = live ? best : INFINITY;
            window(k + 1)[t] = v;
            if (b < B) {
                if (last) a.F_out[b] = v;
                else publish(k, v, mn.x, mc.y);
            }
            int32_t wo = -1;
            const int32_t who = active ? point(k, best, idx, dense, t, wo) : -1;
            if (b < B) {
                a.bp[(int64_t)k * B + b] = live ? who : -1;
                if (a.bp_off) a.bp_off[(int64_t)k * B + b] = live ? wo : -1;
            }
        } else if (!last) {
            // chunk c + 1 replaces chunk c - 1 once step cMC - 1 has read its metadata
            if ((k + 1) % MC == 0) load_meta((k + 1) / MC + 1);
            // Bring the next step's table into the scalar cache, where the dense scan
            // reads it: the first and last entry of each group of 8.  A wave's first
            // group is touched before the staging and consumed after it, so the loads
            // fly meanwhile; further groups (offset ranges above 12 groups) follow.
            const bool touch = dense_step(mn) && b0 < mn.y;
            const_f64 *et = (const_f64 *)(w.ebits + mn.z);
            const int ng = (mn.x + 8) / 8, g0 = ws / 64;
            double e0 = 0.0, e7 = 0.0;
            if (touch && g0 < ng) {
                e0 = et[8 * g0];
                e7 = et[8 * g0 + 7];
            }
            if (moves) stage(k + 1, mn, mc.y);
            asm volatile("" ::"s"(e0), "s"(e7));
            if (touch) {
                for (int g = g0 + NS / 64; g < ng; g += NS / 64) {
                    const double f0 = et[8 * g], f7 = et[8 * g + 7];
                    asm volatile("" ::"s"(f0), "s"(f7));
                }
            }
        }
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

// Bins whose value is strictly below every earlier bin, in three passes over chunks of
// KR_ST_CHUNK bins, one block each: the least value of every chunk; then per chunk the
// least value before it (from the chunk minima), a prefix-minimum scan inside it and
// its count of kept bins; then the output position from the counts before it, and the
// writes.  Thread t holds bins 4t .. 4t + 3 of its chunk.
#define KR_ST_NT 256

__device__ __forceinline__ double st_bin(const ComposeArgs &a, int b)
{
    return b < a.B ? a.F_out[b] : INFINITY;
}

__global__ void __launch_bounds__(KR_ST_NT) staircase_min_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ double sm[KR_ST_NT / 64];
    const int base = blockIdx.x * KR_ST_CHUNK;
    double m = INFINITY;
#pragma unroll
    for (int q = 0; q < KR_ST_CHUNK / KR_ST_NT; ++q)
        m = MinF64()(m, st_bin(a, base + q * KR_ST_NT + threadIdx.x));
    double tot;
    block_scan_excl<KR_ST_NT>(m, (double)INFINITY, MinF64(), sm, &tot);
    if (threadIdx.x == 0) w.chmin[blockIdx.x] = tot;
}

// Least value before this chunk, and this thread's kept bins (bit q: bin 4t + q).
__device__ __forceinline__ uint32_t st_keep(const ComposeArgs &a, const ComposeWs &w,
                                            double *sm, double (&v)[4])
{
    double before = INFINITY;
    for (int c = threadIdx.x; c < (int)blockIdx.x; c += KR_ST_NT)
        before = MinF64()(before, w.chmin[c]);
    double tot;
    block_scan_excl<KR_ST_NT>(before, (double)INFINITY, MinF64(), sm, &tot);
    const int b0 = blockIdx.x * KR_ST_CHUNK + 4 * threadIdx.x;
    double tm = INFINITY;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v[q] = st_bin(a, b0 + q);
        tm = MinF64()(tm, v[q]);
    }
    double run = block_scan_excl<KR_ST_NT>(tm, (double)INFINITY, MinF64(), sm, &before);
    run = MinF64()(run, tot);
    uint32_t k = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (v[q] < run) {
            k |= 1u << q;
            run = v[q];
        }
    return k;
}

__global__ void __launch_bounds__(KR_ST_NT) staircase_count_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ double sm[KR_ST_NT / 64];
    __shared__ int32_t si[KR_ST_NT / 64];
    double v[4];
    const uint32_t k = st_keep(a, w, sm, v);
    int32_t n;
    block_scan_excl<KR_ST_NT>((int32_t)__popc(k), 0, SumI32(), si, &n);
    if (threadIdx.x == 0) w.chcnt[blockIdx.x] = n;
}

__global__ void __launch_bounds__(KR_ST_NT) staircase_write_kernel(ComposeArgs a, ComposeWs w)
{
    __shared__ double sm[KR_ST_NT / 64];
    __shared__ int32_t si[KR_ST_NT / 64];
    const int nb = gridDim.x;
    int32_t before = 0, all = 0;
    for (int c = threadIdx.x; c < nb; c += KR_ST_NT) {
        const int32_t x = w.chcnt[c];
        if (c < (int)blockIdx.x) before += x;
        all += x;
    }
    int32_t tb, ta;
    block_scan_excl<KR_ST_NT>(before, 0, SumI32(), si, &tb);
    block_scan_excl<KR_ST_NT>(all, 0, SumI32(), si, &ta);
    double v[4];
    const uint32_t k = st_keep(a, w, sm, v);
    int32_t n;
    int32_t pos = tb + block_scan_excl<KR_ST_NT>((int32_t)__popc(k), 0, SumI32(), si, &n);
    const double delta = a.info[0], tmin_sum = a.info[1];
    const int b0 = blockIdx.x * KR_ST_CHUNK + 4 * threadIdx.x;
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (k >> q & 1u) {
            a.stair_bin[pos] = b0 + q;
            a.stair_Tlo[pos] = tmin_sum + (double)(b0 + q) * delta;
            a.stair_E[pos] = v[q];
            ++pos;
        }
    // a composition that failed (status set by an earlier kernel) has no staircase
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.n_stair = *a.status == KR_OK ? ta : 0;
}

hipError_t launch_compose(const ComposeArgs &a, const ComposeWs &w, hipEvent_t *minplus_ev,
                          hipStream_t st)
{
    hipLaunchKernelGGL(compose_init_kernel, dim3(1), dim3(64), 0, st, a, w);
    hipLaunchKernelGGL(compose_range_kernel, dim3(a.P), dim3(KR_BLOCK), 0, st, a, w);
    hipLaunchKernelGGL(compose_setup_kernel, dim3(1), dim3(KR_BLOCK), 0, st, a, w);
    hipLaunchKernelGGL(compose_bin_fill_kernel, dim3(2 * a.P - 1), dim3(KR_BLOCK), 0, st, a, w);
    const int G = (a.B + KR_MP_W - 1) / KR_MP_W;
    if (minplus_ev) (void)hipEventRecord(minplus_ev[0], st);
    hipLaunchKernelGGL(minplus_wavefront_kernel, dim3(G), dim3(KR_MP_W * KR_MP_Q), 0, st, a, w);
    if (minplus_ev) (void)hipEventRecord(minplus_ev[1], st);
    {
        const int nb = (a.B + KR_ST_CHUNK - 1) / KR_ST_CHUNK;
        hipLaunchKernelGGL(staircase_min_kernel, dim3(nb), dim3(KR_ST_NT), 0, st, a, w);
        hipLaunchKernelGGL(staircase_count_kernel, dim3(nb), dim3(KR_ST_NT), 0, st, a, w);
        hipLaunchKernelGGL(staircase_write_kernel, dim3(nb), dim3(KR_ST_NT), 0, st, a, w);
    }
    return hipGetLastError();
}

// Walk the back-pointers of each query bin from the last partition to the first; one
// wave per query.  A step needs the chosen point's offset (a load that depends on the
// back-pointer) and then the next back-pointer (a load that depends on the offset).  The
// wave loads the next row's back-pointers for the KR_EX_SPEC bins just below the current
// one while the offset is in flight, so a step costs one memory latency when the offset
// is below KR_EX_SPEC (else one more load).  With ST (at most KR_EX_LP partitions) the
// partition offsets are staged in LDS first and the choices are kept there until the
// walk ends, so no step waits for an offset load or for a store.
#define KR_EX_SPEC 128
#define KR_EX_RS 2048  // partitions per pass of the final sums
#define KR_EX_LP 2048  // most partitions whose offsets and choices the walk keeps in LDS

template <bool ST>
__global__ void __launch_bounds__(64) extract_kernel(ExtractArgs a)
{
    __shared__ double sT[KR_EX_RS], sE[KR_EX_RS];
    __shared__ int64_t s_off[ST ? KR_EX_LP + 1 : 1];
    __shared__ int32_t s_ch[ST ? KR_EX_LP : 1];
    const int P = a.P;
    const int q = blockIdx.x, lane = threadIdx.x;
    int32_t *choice = a.choice + (int64_t)q * a.P;
    auto off_at = [&](int k) -> int64_t {
        if constexpr (ST) return s_off[k];
        else return a.off[k];
    };
    if constexpr (ST) {
        for (int k = lane; k <= P; k += 64) s_off[k] = a.off[k];
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
        __builtin_amdgcn_s_waitcnt(0xC07F);
    }
    int64_t b = a.bins[q];
    bool ok = b >= 0 && b < a.B;
    int32_t j = ok ? a.bp[(int64_t)(a.P - 1) * a.B + b] : -1;
    int64_t lo = off_at(P - 1), hi = off_at(P);
    for (int k = a.P - 1; k >= 0 && ok; --k) {
        const int64_t n = hi - lo;
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
        if constexpr (ST) {
            if (lane == 0) s_ch[k] = j;
        } else {
            if (lane == 0) choice[k] = j;
        }
        if (k > 0) {  // the next partition's offsets, while the loads are in flight
            hi = lo;
            lo = off_at(k - 1);
        }
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
    // Exact T and E of the choice: the lanes gather the chosen points' values into LDS,
    // one lane adds them in partition order.
    if constexpr (ST) {
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
        __builtin_amdgcn_s_waitcnt(0xC07F);
    } else {
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's choice stores are done
    }
    double Ts = 0.0, Es = 0.0;
    for (int k0 = 0; k0 < P; k0 += KR_EX_RS) {
        const int kn = min(P - k0, KR_EX_RS);
        for (int i = lane; i < kn; i += 64) {
            const int kk = k0 + i;
            if (ok) {
                int32_t c;
                if constexpr (ST) {
                    c = s_ch[kk];
                    choice[kk] = c;
                } else {
                    c = load_l2(choice + kk);
                }
                const int64_t x = off_at(kk) + c;
                sT[i] = a.T[x];
                sE[i] = a.E[x];
                if (a.cand_idx) a.choice_cand[(int64_t)q * P + kk] = a.cand_idx[x];
            } else {
                choice[kk] = -1;
                if (a.cand_idx) a.choice_cand[(int64_t)q * P + kk] = -1;
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
        __builtin_amdgcn_s_waitcnt(0xC07F);
        if (ok && lane == 0)
            for (int i = 0; i < kn; ++i) {
                Ts = Ts + sT[i];
                Es = Es + sE[i];
            }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
        __builtin_amdgcn_s_waitcnt(0xC07F);
    }
    if (lane != 0) return;
    a.T_out[q] = ok ? Ts : NAN;
    a.E_out[q] = ok ? Es : NAN;
    a.ok[q] = ok;
}

// Walk over the recorded offsets (bp_off): the bin of row k - 1 is b - bp_off[k][b], so a
// step needs one table entry and no point lookup.  The wave keeps windows of the next
// KR_XW_D rows in registers: slot d holds KR_XW_W consecutive bins of its row (lane l
// the 8 bins from base + 8 l), loaded KR_XW_D steps before the row is walked, so the
// loads fly meanwhile.  A window is placed where the offsets of the last KR_XW_D rows put
// that row's bin; a bin outside its window is loaded directly.  The bins of all rows are
// kept in LDS, and the chosen points are gathered from bp afterwards, all rows at once.
// At most KR_EX_LP partitions and KR_XW_MAX table entries (32-bit byte offsets).
#define KR_XW_D 16   // rows of look-ahead
#define KR_XW_W 512  // bins per window (8 per lane)
#define KR_XW_MAX (1 << 29)
typedef int32_t i32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));  // 4-byte aligned

// f where the wave-uniform mask m is 0, t where it is all ones (one VALU select; the
// compiler would branch on the uniform condition instead)
__device__ __forceinline__ int32_t kr_usel(int32_t f, int32_t t, uint64_t m)
{
    int32_t r;
    asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(f), "v"(t), "s"(m));
    return r;
}

// v with lane L set to the wave-uniform s
template <int L>
__device__ __forceinline__ int32_t kr_setlane(int32_t v, int32_t s)
{
    asm("v_writelane_b32 %0, %1, %2" : "+v"(v) : "s"(s), "I"(L));
    return v;
}

// f(std::integral_constant<int, I>) for I = 0 .. N - 1, in order, unrolled
template <typename F, int... I>
__device__ __forceinline__ void kr_unroll(F &&f, std::integer_sequence<int, I...>)
{
    (f(std::integral_constant<int, I>{}), ...);
}

__global__ void __launch_bounds__(64) extract_walk_kernel(ExtractArgs a)
{
    __shared__ double sT[KR_EX_RS], sE[KR_EX_RS];
    __shared__ int64_t s_off[KR_EX_LP + 1];
    __shared__ int32_t s_b[KR_EX_LP];
    __shared__ int32_t s_ch[KR_EX_LP];
    constexpr int D = KR_XW_D, W = KR_XW_W;
    const int P = a.P;
    const int32_t B = a.B;
    const int32_t total = P * B;  // at most KR_XW_MAX
    const int q = blockIdx.x, lane = threadIdx.x;
    int32_t *choice = a.choice + (int64_t)q * P;
    for (int k = lane; k <= P; k += 64) s_off[k] = a.off[k];

    i32x4_a4 wl[D], wh[D];  // slot d: bins base[d] + 8 lane + 0..3, + 4..7 of its row
    int32_t base[D];
    // window of the row starting at table index r0, placed below bin bk by the predicted
    // drift (a guess: any value works), then moved to lie inside the table (it holds at
    // least W entries): entries that run into a neighbouring row are never read, since a
    // walk's bins stay in [0, B)
    auto issue = [&](int d, int32_t r0, int32_t bk, int32_t drift) {
        int32_t x0 = r0 + min(bk - drift - W / 2, bk - (W - 1));
        x0 = min(max(x0, 0), total - W);
        base[d] = x0 - r0;
        const uint32_t x = (uint32_t)(x0 + 8 * lane);
        wl[d] = *(const i32x4_a4 *)(a.bp_off + x);
        wh[d] = *(const i32x4_a4 *)(a.bp_off + x + 4);
    };
    // the recorded offset at bin bk of the row starting at r0: from slot d when bk is in
    // its window, else loaded
    auto lookup = [&](int d, int32_t r0, int32_t bk) -> int32_t {
        const int32_t pos = bk - base[d];
        const uint64_t m2 = (pos & 4) ? ~0ull : 0ull, m1 = (pos & 2) ? ~0ull : 0ull,
                       m0 = (pos & 1) ? ~0ull : 0ull;
        const int32_t y0 = kr_usel(wl[d].x, wh[d].x, m2), y1 = kr_usel(wl[d].y, wh[d].y, m2);
        const int32_t y2 = kr_usel(wl[d].z, wh[d].z, m2), y3 = kr_usel(wl[d].w, wh[d].w, m2);
        const int32_t z0 = kr_usel(y0, y2, m1), z1 = kr_usel(y1, y3, m1);
        int32_t o = __builtin_amdgcn_readlane(kr_usel(z0, z1, m0), (pos >> 3) & 63);
        if (__builtin_expect((uint32_t)pos >= (uint32_t)W, 0)) o = a.bp_off[r0 + bk];
        return o;
    };

    const int32_t b_query = a.bins[q];
    int32_t b = b_query;
    bool ok = b >= 0 && b < B;
    if (!ok) b = 0;  // walked anyway (the results are discarded)
    // drift predicted for D rows: the offsets of the last D rows (to start with, the
    // query bin spread over all rows)
    int32_t hist[D];  // the bin D rows back, by slot
    const int32_t avg0 = b / max(P, 1);
#pragma unroll
    for (int d = 0; d < D; ++d) {
        hist[d] = b;
        issue(d, max(P - 1 - d, 0) * B, b, d * avg0);
    }
    // lane d holds the bin of row k0 - d of the current block of D rows (top row k0)
    int32_t brow = 0;
    int32_t neg = 0;  // sign bit set once an offset is -1 (no point) or a bin falls below 0
    // one row: take its offset, record its bin, refill its slot with the row D below.  A
    // failed walk goes on from bin 0 (memory-safe) and is dropped at the end.
    auto step = [&](auto dc, int32_t r0) {
        constexpr int d = decltype(dc)::value;
        const int32_t o = lookup(d, r0, b);
        brow = kr_setlane<d>(brow, b);
        const int32_t bn = b - o;
        neg |= o | bn;
        b = max(bn, 0);
        const int32_t drift = hist[d] - b;  // the offsets of the last D rows
        hist[d] = b;
        issue(d, r0 - D * B, b, drift);  // row k - D (clamped into the table)
    };
    int k = P - 1;
    int32_t rk = k * B;
    for (; k >= D - 1; k -= D, rk -= D * B) {
        kr_unroll([&](auto dc) { step(dc, rk - decltype(dc)::value * B); },
                  std::make_integer_sequence<int, D>{});  // row k - d: slot d
        if (lane < D) s_b[k - lane] = brow;
    }
    if (k >= 0) {  // the last rows, fewer than D
        kr_unroll(
            [&](auto dc) {
                if (decltype(dc)::value <= k) step(dc, rk - decltype(dc)::value * B);
            },
            std::make_integer_sequence<int, D - 1>{});
        if (lane <= k) s_b[k - lane] = brow;
    }
    ok = ok && neg >= 0;
    ok = ok && b == 0;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
    __builtin_amdgcn_s_waitcnt(0xC07F);
    // the chosen points, all rows at once
    for (int kk = lane; kk < P; kk += 64) {
        const int32_t c = ok ? a.bp[(int64_t)kk * B + s_b[kk]] : -1;
        s_ch[kk] = c;
        choice[kk] = c;
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
    __builtin_amdgcn_s_waitcnt(0xC07F);
    // exact T and E of the choice: the lanes gather the chosen points' values into LDS,
    // one lane adds them in partition order
    double Ts = 0.0, Es = 0.0;
    for (int k0 = 0; k0 < P; k0 += KR_EX_RS) {
        const int kn = min(P - k0, KR_EX_RS);
        for (int i = lane; i < kn; i += 64) {
            const int kk = k0 + i;
            const int32_t c = s_ch[kk];
            if (ok) {
                const int64_t x = s_off[kk] + c;
                sT[i] = a.T[x];
                sE[i] = a.E[x];
                if (a.cand_idx) a.choice_cand[(int64_t)q * P + kk] = a.cand_idx[x];
            } else if (a.cand_idx) {
                a.choice_cand[(int64_t)q * P + kk] = -1;
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
        __builtin_amdgcn_s_waitcnt(0xC07F);
        if (ok && lane == 0)
            for (int i = 0; i < kn; ++i) {
                Ts = Ts + sT[i];
                Es = Es + sE[i];
            }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
        __builtin_amdgcn_s_waitcnt(0xC07F);
    }
    if (lane != 0) return;
    a.T_out[q] = ok ? Ts : NAN;
    a.E_out[q] = ok ? Es : NAN;
    a.ok[q] = ok;
}

hipError_t launch_extract(const ExtractArgs &a, hipStream_t st)
{
    if (a.n_q == 0) return hipSuccess;
    if (a.bp_off && a.P <= KR_EX_LP && (int64_t)a.P * a.B >= KR_XW_W &&
        (int64_t)a.P * a.B <= KR_XW_MAX)
        hipLaunchKernelGGL(extract_walk_kernel, dim3(a.n_q), dim3(64), 0, st, a);
    else if (a.P <= KR_EX_LP)
        hipLaunchKernelGGL(extract_kernel<true>, dim3(a.n_q), dim3(64), 0, st, a);
    else
        hipLaunchKernelGGL(extract_kernel<false>, dim3(a.n_q), dim3(64), 0, st, a);
    return hipGetLastError();
}

}  // namespace kr
