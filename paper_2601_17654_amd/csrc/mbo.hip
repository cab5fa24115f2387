// Scores and batch selection of the multi-pass Bayesian optimisation (Section 4.3,
// Algorithm 1; reference point from Appendix C).
//
// Exploitation scores.  For each partition and each energy variant (total E, dynamic
// E - p_static * T, static p_static * T) one block turns the measured points into their
// staircase (strictly increasing T, strictly decreasing energy) and its hypervolume
// against r = 1.1 x the worst measured values.  The score kernel then stages a
// partition's three staircases in LDS and gives every candidate y its hypervolume
// improvement directly as the area that y adds: the part of [y.T, rT] x [y.E, rE] that
// no staircase step covers, summed strip by strip from y.T rightwards until a step at or
// below y.E closes it.  That is exact in real arithmetic and never forms the difference
// of two large hypervolumes.
//
// Selection.  Every pass is a top-k by (score descending, index ascending) over the
// partition's unmeasured candidates, with k <= 64.  A wave keeps its best 64 entries
// sorted across its lanes; each batch of 64 new candidates is compared against the
// current 64th entry, and only when one of them beats it is the batch sorted (bitonic,
// lane shuffles) and merged in (reverse, lane-wise better, bitonic merge).  Tiles of a
// partition reduce to one sorted list per pass; one block per partition merges the tile
// lists and assembles the batch in pass order.
#include <math.h>

#include "kr_device.h"
#include "kr_launch.h"

namespace kr {

__device__ __forceinline__ double energy_variant(int v, double t, double e, double ps)
{
    if (v == 0) return e;
    if (v == 1) return e - ps * t;  // no contraction: the library is built without it
    return ps * t;
}

struct HvMaxF64 {
    __device__ __forceinline__ double operator()(double a, double b) const { return b > a ? b : a; }
};
struct SumI32x {
    __device__ __forceinline__ int32_t operator()(int32_t a, int32_t b) const { return a + b; }
};

__global__ void hvi_init_kernel(int32_t *status) { *status = KR_OK; }

// One block per partition: reference point, the three staircases and their HV.
__global__ void __launch_bounds__(KR_BLOCK) hvi_prep_kernel(HviArgs a)
{
    __shared__ double sT[KR_HVI_MAX_OBS], sE[KR_HVI_MAX_OBS], sV[KR_HVI_MAX_OBS];
    __shared__ double fT[KR_HVI_MAX_OBS], fE[KR_HVI_MAX_OBS];
    __shared__ int32_t keep[KR_HVI_MAX_OBS];
    __shared__ double red[KR_WAVES];
    __shared__ int32_t ired[KR_WAVES];
    const int g = blockIdx.x, tid = threadIdx.x;
    const int64_t o0 = a.obs_off[g], no64 = a.obs_off[g + 1] - o0;
    if (no64 < 1 || no64 > KR_HVI_MAX_OBS) {
        if (tid < 3) {
            a.fr_n[g * 3 + tid] = -1;
            a.hv[g * 3 + tid] = NAN;
        }
        if (tid < 4) a.ref[g * 4 + tid] = NAN;
        if (tid == 0) *a.status = KR_EINVAL;
        return;
    }
    const int no = (int)no64;
    double mt = -INFINITY;
    for (int i = tid; i < no; i += KR_BLOCK) {
        sT[i] = a.T_obs[o0 + i];
        sE[i] = a.E_obs[o0 + i];
        mt = sT[i] > mt ? sT[i] : mt;
    }
    const double rT = 1.1 * block_reduce(mt, (double)-INFINITY, HvMaxF64(), red);
    if (tid == 0) a.ref[g * 4] = rT;
    for (int v = 0; v < 3; ++v) {
        double me = -INFINITY;
        for (int i = tid; i < no; i += KR_BLOCK) {
            sV[i] = energy_variant(v, sT[i], sE[i], a.p_static);
            me = sV[i] > me ? sV[i] : me;
        }
        const double rE = 1.1 * block_reduce(me, (double)-INFINITY, HvMaxF64(), red);
        // a point opens a staircase step iff it is inside the box and no point inside the
        // box is at least as good in both and earlier in (T, energy, index) order
        int32_t mine = 0;
        for (int i = tid; i < no; i += KR_BLOCK) {
            const double ti = sT[i], ei = sV[i];
            bool k = ti < rT && ei < rE;
            for (int j = 0; j < no && k; ++j) {
                const double tj = sT[j], ej = sV[j];
                if (j != i && tj < rT && ej < rE && tj <= ti && ej <= ei &&
                    (tj < ti || ej < ei || j < i))
                    k = false;
            }
            keep[i] = k;
            mine += k;
        }
        const int32_t s = block_reduce(mine, 0, SumI32x(), ired);
        // rank = steps with smaller time (step times are distinct)
        for (int i = tid; i < no; i += KR_BLOCK) {
            if (!keep[i]) continue;
            int r = 0;
            for (int j = 0; j < no; ++j) r += keep[j] && sT[j] < sT[i];
            fT[r] = sT[i];
            fE[r] = sV[i];
            a.fr_T[(int64_t)v * a.n_obs + o0 + r] = sT[i];
            a.fr_E[(int64_t)v * a.n_obs + o0 + r] = sV[i];
        }
        __syncthreads();
        if (tid == 0) {
            double hv = 0.0;
            for (int r = 0; r < s; ++r) {
                const double next = r + 1 < s ? fT[r + 1] : rT;
                hv = hv + (next - fT[r]) * (rE - fE[r]);
            }
            a.hv[g * 3 + v] = hv;
            a.ref[g * 4 + 1 + v] = rE;
            a.fr_n[g * 3 + v] = s;
        }
        __syncthreads();
    }
}

// Area that y = (t, e) adds to the staircase (fT, fE)[0, s) inside the box below (rT, rE).
__device__ __forceinline__ double hvi_one(const double *fT, const double *fE, int s, double rT,
                                          double rE, double t, double e)
{
    if (!(t < rT) || !(e < rE)) return 0.0;
    int lo = 0, hi = s;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (fT[mid] <= t) lo = mid + 1;
        else hi = mid;
    }
    double level = lo == 0 ? rE : fE[lo - 1];
    if (level <= e) return 0.0;  // a step at or before t is at or below e
    double area = 0.0, start = t;
    int i = lo;
    while (i < s && fE[i] > e) {
        area = area + (fT[i] - start) * (level - e);
        start = fT[i];
        level = fE[i];
        ++i;
    }
    const double end = i < s ? fT[i] : rT;
    return area + (end - start) * (level - e);
}

// Flat tiles of KR_HVI_TILE candidates; a tile visits every partition it overlaps.
__global__ void __launch_bounds__(KR_BLOCK) hvi_score_kernel(HviArgs a)
{
    __shared__ double fT[3][KR_HVI_MAX_OBS], fE[3][KR_HVI_MAX_OBS];
    const int tid = threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.x * KR_HVI_TILE;
    const int64_t t1 = t0 + KR_HVI_TILE < a.n_cand ? t0 + KR_HVI_TILE : a.n_cand;
    // last partition starting at or before t0 (uniform binary search)
    int lo = 0, hi = a.n_seg;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (a.cand_off[mid] <= t0) lo = mid;
        else hi = mid;
    }
    for (int g = lo; g < a.n_seg && a.cand_off[g] < t1; ++g) {
        const int64_t c0 = a.cand_off[g], c1 = a.cand_off[g + 1];
        if (c1 <= t0) continue;
        const int64_t o0 = a.obs_off[g];
        int s[3];
        bool bad = false;
        for (int v = 0; v < 3; ++v) {
            s[v] = a.fr_n[g * 3 + v];
            bad = bad || s[v] < 0;
        }
        __syncthreads();
        if (!bad)
            for (int v = 0; v < 3; ++v)
                for (int i = tid; i < s[v]; i += KR_BLOCK) {
                    fT[v][i] = a.fr_T[(int64_t)v * a.n_obs + o0 + i];
                    fE[v][i] = a.fr_E[(int64_t)v * a.n_obs + o0 + i];
                }
        __syncthreads();
        const double rT = a.ref[g * 4];
        const double rE[3] = {a.ref[g * 4 + 1], a.ref[g * 4 + 2], a.ref[g * 4 + 3]};
        const int64_t x0 = c0 > t0 ? c0 : t0, x1 = c1 < t1 ? c1 : t1;
        // all of this thread's candidates of the partition are loaded before any is
        // scored, so their loads are in flight together
        constexpr int kPer = KR_HVI_TILE / KR_BLOCK;
        double t[kPer], e[kPer];
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int64_t x = x0 + tid + (int64_t)j * KR_BLOCK;
            t[j] = x < x1 ? __builtin_nontemporal_load(a.T_hat + x) : 0.0;
            e[j] = x < x1 ? __builtin_nontemporal_load(a.E_hat + x) : 0.0;
        }
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int64_t x = x0 + tid + (int64_t)j * KR_BLOCK;
            if (x >= x1) break;
#pragma unroll
            for (int v = 0; v < 3; ++v) {
                const double h = bad ? NAN
                                     : hvi_one(fT[v], fE[v], s[v], rT, rE[v], t[j],
                                               energy_variant(v, t[j], e[j], a.p_static));
                __builtin_nontemporal_store(h, a.hvi + (int64_t)v * a.n_cand + x);
            }
        }
    }
}

// ev: optional start/stop events around the score kernel (null entries: none).
static void mark(hipEvent_t *ev, int which, hipStream_t st)
{
    if (ev && ev[0] && ev[1]) (void)hipEventRecord(ev[which], st);
}

hipError_t launch_hvi(const HviArgs &a, hipEvent_t *ev, hipStream_t st)
{
    hipLaunchKernelGGL(hvi_init_kernel, dim3(1), dim3(1), 0, st, a.status);
    hipLaunchKernelGGL(hvi_prep_kernel, dim3(a.n_seg), dim3(KR_BLOCK), 0, st, a);
    if (a.n_cand > 0) {
        const int64_t blocks = (a.n_cand + KR_HVI_TILE - 1) / KR_HVI_TILE;
        mark(ev, 0, st);
        hipLaunchKernelGGL(hvi_score_kernel, dim3((unsigned)blocks), dim3(KR_BLOCK), 0, st, a);
        mark(ev, 1, st);
    }
    return hipGetLastError();
}

// Population standard deviation of the members' T plus that of their E.  With M a
// compile-time count the members stay in registers between the mean and the deviations;
// the generic form reads them twice.
template <int MC>
__global__ void __launch_bounds__(KR_BLOCK) unc_kernel(int M_rt, int64_t n, const double *Tm,
                                                     const double *Em, double *unc)
{
    const int M = MC > 0 ? MC : M_rt;
    const int64_t stride = (int64_t)gridDim.x * KR_BLOCK;
    if constexpr (MC > 0) {
        // two candidates per step, all their members loaded before either is reduced
        for (int64_t x = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x; x < n; x += 2 * stride) {
            const int64_t xs[2] = {x, x + stride < n ? x + stride : x};
            double t[2][MC], e[2][MC];
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int m = 0; m < MC; ++m) {
                    t[j][m] = __builtin_nontemporal_load(Tm + (int64_t)m * n + xs[j]);
                    e[j][m] = __builtin_nontemporal_load(Em + (int64_t)m * n + xs[j]);
                }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                double st = 0.0, se = 0.0;
#pragma unroll
                for (int m = 0; m < MC; ++m) {
                    st = st + t[j][m];
                    se = se + e[j][m];
                }
                const double mt = st / M, me = se / M;
                double vt = 0.0, ve = 0.0;
#pragma unroll
                for (int m = 0; m < MC; ++m) {
                    const double dt = t[j][m] - mt, de = e[j][m] - me;
                    vt = vt + dt * dt;
                    ve = ve + de * de;
                }
                if (j == 0 || x + stride < n)
                    __builtin_nontemporal_store(sqrt(vt / M) + sqrt(ve / M), unc + xs[j]);
            }
        }
        return;
    }
    for (int64_t x = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x; x < n; x += stride) {
        double st = 0.0, se = 0.0;
        {
            for (int m = 0; m < M; ++m) {
                st = st + Tm[(int64_t)m * n + x];
                se = se + Em[(int64_t)m * n + x];
            }
            const double mt = st / M, me = se / M;
            double vt = 0.0, ve = 0.0;
            for (int m = 0; m < M; ++m) {
                const double dt = Tm[(int64_t)m * n + x] - mt, de = Em[(int64_t)m * n + x] - me;
                vt = vt + dt * dt;
                ve = ve + de * de;
            }
            unc[x] = sqrt(vt / M) + sqrt(ve / M);
        }
    }
}

hipError_t launch_uncertainty(int M, int64_t n, const double *Tm, const double *Em, double *unc,
                              hipEvent_t *ev, hipStream_t st)
{
    if (n == 0) return hipSuccess;
    const int64_t blocks = (n + KR_BLOCK - 1) / KR_BLOCK;
    const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
    const dim3 g(grid), b(KR_BLOCK);
    mark(ev, 0, st);
    switch (M) {
    case 1: hipLaunchKernelGGL(unc_kernel<1>, g, b, 0, st, M, n, Tm, Em, unc); break;
    case 2: hipLaunchKernelGGL(unc_kernel<2>, g, b, 0, st, M, n, Tm, Em, unc); break;
    case 3: hipLaunchKernelGGL(unc_kernel<3>, g, b, 0, st, M, n, Tm, Em, unc); break;
    case 4: hipLaunchKernelGGL(unc_kernel<4>, g, b, 0, st, M, n, Tm, Em, unc); break;
    case 5: hipLaunchKernelGGL(unc_kernel<5>, g, b, 0, st, M, n, Tm, Em, unc); break;
    case 6: hipLaunchKernelGGL(unc_kernel<6>, g, b, 0, st, M, n, Tm, Em, unc); break;
    case 7: hipLaunchKernelGGL(unc_kernel<7>, g, b, 0, st, M, n, Tm, Em, unc); break;
    case 8: hipLaunchKernelGGL(unc_kernel<8>, g, b, 0, st, M, n, Tm, Em, unc); break;
    default: hipLaunchKernelGGL(unc_kernel<0>, g, b, 0, st, M, n, Tm, Em, unc); break;
    }
    mark(ev, 1, st);
    return hipGetLastError();
}

// ---- selection -----------------------------------------------------------------------

// Order key of a score: larger key = larger score; -0 and +0 share one key.  Key 0 is
// below every score and marks an empty list entry.
__device__ __forceinline__ uint64_t score_key(double s)
{
    if (s == 0.0) s = 0.0;
    const uint64_t u = dbits(s);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

struct Entry {
    uint64_t key;
    int32_t idx;
};

__device__ __forceinline__ bool better(const Entry &a, const Entry &b)
{
    return a.key > b.key || (a.key == b.key && a.idx < b.idx);
}

__device__ __forceinline__ Entry shfl_entry(const Entry &e, int src)
{
    Entry r;
    const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)e.key, src, 64);
    const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(e.key >> 32), src, 64);
    r.key = ((uint64_t)hi << 32) | lo;
    r.idx = __shfl(e.idx, src, 64);
    return r;
}

// One compare-exchange step with lane ^ j; `up` lanes keep the better entry of the pair
// when they are the lower lane of it.
__device__ __forceinline__ Entry cmpx(const Entry &e, int lane, int j, bool up)
{
    const Entry p = shfl_entry(e, lane ^ j);
    const bool lower = (lane & j) == 0;
    const bool take = lower == up ? better(p, e) : better(e, p);
    return take ? p : e;
}

// Sort a wave's 64 entries best first.
__device__ __forceinline__ Entry wave_sort(Entry e, int lane)
{
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) e = cmpx(e, lane, j, (lane & k) == 0 || k == 64);
    return e;
}

// Best 64 of two best-first lists, best first.
__device__ __forceinline__ Entry wave_merge(const Entry &list, const Entry &sorted, int lane)
{
    const Entry r = shfl_entry(sorted, 63 - lane);
    Entry e = better(list, r) ? list : r;
#pragma unroll
    for (int j = 32; j > 0; j >>= 1) e = cmpx(e, lane, j, true);
    return e;
}

// Offer one entry per lane to the list.
__device__ __forceinline__ Entry wave_offer(const Entry &list, Entry c, int lane)
{
    Entry worst;
    worst.key = lane_u64(list.key, 63);
    worst.idx = lane_i32(list.idx, 63);
    if (!better(c, worst)) {
        c.key = 0;
        c.idx = INT32_MAX;
    }
    if (__ballot(c.key != 0) == 0) return list;
    return wave_merge(list, wave_sort(c, lane), lane);
}

// tile_off[g] = first selection tile of partition g; clears the NaN flag.  One block.
__global__ void __launch_bounds__(KR_BLOCK) sel_plan_kernel(SelArgs a)
{
    __shared__ int64_t red[KR_WAVES];
    int64_t carry = 0;
    for (int64_t base = 0; base < a.n_seg; base += KR_BLOCK) {
        const int64_t g = base + threadIdx.x;
        const int64_t n = g < a.n_seg ? a.cand_off[g + 1] - a.cand_off[g] : 0;
        const int64_t tiles = (n + KR_SEL_TILE - 1) / KR_SEL_TILE;
        int64_t total;
        const int64_t ex = block_exclusive(tiles, (int64_t)0, SumI64(), red, &total);
        if (g < a.n_seg) a.tile_off[g] = carry + ex;
        carry += total;
    }
    if (threadIdx.x == 0) {
        a.tile_off[a.n_seg] = carry;
        *a.flag = 0;
    }
}

// One block per tile: each pass's best KR_SEL_LIST unmeasured candidates of the tile, in
// one sweep over the scores of all passes.  Per pass a wave keeps its sorted list and a
// threshold (the list's last entry); candidates that beat the threshold are compacted
// into an LDS buffer, and the buffer is sorted and merged into the list only when the
// next batch would overflow it, so merges grow with the log of the candidates seen
// rather than with their number.
__global__ void __launch_bounds__(KR_BLOCK) sel_tile_kernel(SelArgs a)
{
    __shared__ uint32_t excl[KR_SEL_TILE / 32];
    __shared__ uint64_t bkey[KR_WAVES][4][KR_SEL_LIST];
    __shared__ int32_t bidx[KR_WAVES][4][KR_SEL_LIST];
    const int64_t b = blockIdx.x;
    if (b >= a.tile_off[a.n_seg]) return;
    int lo = 0, hi = a.n_seg;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (a.tile_off[mid] <= b) lo = mid;
        else hi = mid;
    }
    const int g = lo;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t c0 = a.cand_off[g], ng = a.cand_off[g + 1] - c0;
    const int64_t l0 = (b - a.tile_off[g]) * KR_SEL_TILE;  // local index of the tile start
    const int64_t l1 = l0 + KR_SEL_TILE < ng ? l0 + KR_SEL_TILE : ng;
    for (int i = tid; i < KR_SEL_TILE / 32; i += KR_BLOCK) excl[i] = 0;
    __syncthreads();
    for (int64_t i = a.obs_off[g] + tid; i < a.obs_off[g + 1]; i += KR_BLOCK) {
        const int64_t x = a.obs_idx[i];
        if (x >= l0 && x < l1) atomicOr(&excl[(x - l0) >> 5], 1u << ((x - l0) & 31));
    }
    __syncthreads();
    const int np = a.npass;
    const double *src[4];
#pragma unroll
    for (int p = 0; p < 4; ++p)
        src[p] = (p < 3 ? a.score + (int64_t)p * a.n_cand : (p < np ? a.unc : a.score)) + c0;
    Entry L[4];
    Entry thr[4];
    int cnt[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        L[p].key = 0;
        L[p].idx = INT32_MAX;
        thr[p] = L[p];
        cnt[p] = 0;
    }
    constexpr int kPerWave = KR_SEL_TILE / KR_WAVES;
    constexpr int kRows = kPerWave / 64, kRowBits = __builtin_ctz(kRows);
    static_assert((kRows & (kRows - 1)) == 0, "rows per wave must be a power of two");
    const int64_t w0 = l0 + (int64_t)wave * kPerWave;  // this wave's first local index
    // Rows of 64 candidates are visited in bit-reversed order.  Scores trend along the
    // index (it runs over frequencies slowest), and in index order late rows would keep
    // beating the list's last entry and force merges; the result does not depend on the
    // order, since (score, index) is a total order.
    auto row = [&](int r) { return w0 + (int64_t)(__brev((uint32_t)r) >> (32 - kRowBits)) * 64 + lane; };
    bool nan_seen = false;
    double cur[4], nxt[4];
    int64_t xn = row(0);
#pragma unroll
    for (int p = 0; p < 4; ++p) cur[p] = p < np && xn < l1 ? __builtin_nontemporal_load(src[p] + xn) : 0.0;
    for (int r = 0; r < kRows; ++r) {
        const int64_t x = xn;
        xn = row(r + 1 < kRows ? r + 1 : r);
#pragma unroll
        for (int p = 0; p < 4; ++p)
            nxt[p] = p < np && r + 1 < kRows && xn < l1 ? __builtin_nontemporal_load(src[p] + xn) : 0.0;
        const int64_t off = x - l0;
        const bool in = x < l1 && !((excl[(off >> 5) & (KR_SEL_TILE / 32 - 1)] >> (off & 31)) & 1u);
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            if (p >= np) break;
            const double v = cur[p];
            nan_seen = nan_seen || (x < l1 && v != v);
            Entry c;
            c.key = in && v == v ? score_key(v) : 0;
            c.idx = (int32_t)x;
            bool pass = c.key != 0 && better(c, thr[p]);
            uint64_t m = __ballot(pass);
            if (m == 0) continue;
            int n = __popcll(m);
            if (cnt[p] + n > KR_SEL_LIST) {
                Entry e;
                e.key = lane < cnt[p] ? bkey[wave][p][lane] : 0;
                e.idx = lane < cnt[p] ? bidx[wave][p][lane] : INT32_MAX;
                L[p] = wave_merge(L[p], wave_sort(e, lane), lane);
                thr[p].key = lane_u64(L[p].key, 63);
                thr[p].idx = lane_i32(L[p].idx, 63);
                cnt[p] = 0;
                pass = c.key != 0 && better(c, thr[p]);
                m = __ballot(pass);
                n = __popcll(m);
            }
            if (pass) {
                const int pos = cnt[p] + (int)__builtin_amdgcn_mbcnt_hi(
                                             (uint32_t)(m >> 32),
                                             __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
                bkey[wave][p][pos] = c.key;
                bidx[wave][p][pos] = c.idx;
            }
            cnt[p] += n;
        }
#pragma unroll
        for (int p = 0; p < 4; ++p) cur[p] = nxt[p];
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        if (p >= np) break;
        if (cnt[p] > 0) {
            Entry e;
            e.key = lane < cnt[p] ? bkey[wave][p][lane] : 0;
            e.idx = lane < cnt[p] ? bidx[wave][p][lane] : INT32_MAX;
            L[p] = wave_merge(L[p], wave_sort(e, lane), lane);
        }
    }
    __syncthreads();  // every wave is done with its buffers
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        if (p >= np) break;
        bkey[wave][p][lane] = L[p].key;
        bidx[wave][p][lane] = L[p].idx;
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            if (p >= np) break;
            Entry list = L[p];
            for (int w = 1; w < KR_WAVES; ++w) {
                Entry o;
                o.key = bkey[w][p][lane];
                o.idx = bidx[w][p][lane];
                list = wave_merge(list, o, lane);
            }
            const int64_t slot = (b * np + p) * KR_SEL_LIST + lane;
            a.part_key[slot] = list.key;
            a.part_idx[slot] = list.idx;
        }
    }
    if (nan_seen) *a.flag = 1;
}

// One block per partition: merge its tile lists per pass and assemble the batch.
__global__ void __launch_bounds__(KR_BLOCK) sel_final_kernel(SelArgs a)
{
    __shared__ uint64_t lkey[4][KR_WAVES][KR_SEL_LIST];
    __shared__ int32_t lidx[4][KR_WAVES][KR_SEL_LIST];
    const int g = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool bad = *a.flag != 0;
    if (g == 0 && tid == 0) *a.status = bad ? KR_EINVAL : KR_OK;
    if (bad) {
        if (tid == 0) a.count[g] = 0;
        return;
    }
    const int64_t tb = a.tile_off[g], te = a.tile_off[g + 1];
    for (int p = 0; p < a.npass; ++p) {
        Entry list;
        list.key = 0;
        list.idx = INT32_MAX;
        for (int64_t t = tb + wave; t < te; t += KR_WAVES) {
            const int64_t slot = (t * a.npass + p) * KR_SEL_LIST + lane;
            Entry o;
            o.key = a.part_key[slot];
            o.idx = a.part_idx[slot];
            list = wave_merge(list, o, lane);
        }
        lkey[p][wave][lane] = list.key;
        lidx[p][wave][lane] = list.idx;
    }
    __syncthreads();
    if (wave != 0) return;
    Entry L[4];
    for (int p = 0; p < a.npass; ++p) {
        Entry list;
        list.key = lkey[p][0][lane];
        list.idx = lidx[p][0][lane];
        for (int w = 1; w < KR_WAVES; ++w) {
            Entry o;
            o.key = lkey[p][w][lane];
            o.idx = lidx[p][w][lane];
            list = wave_merge(list, o, lane);
        }
        L[p] = list;
    }
    // the batch: lane i holds its i-th member
    int32_t mine = -1;
    int cnt = 0;
    const int k = a.k[3];
    for (int p = 0; p < a.npass; ++p) {
        const int want = p < 3 ? a.k[p] : KR_SEL_LIST;
        for (int r = 0; r < want && cnt < (p < 3 ? KR_SEL_LIST : k); ++r) {
            const uint64_t key = lane_u64(L[p].key, r);
            if (key == 0) break;
            const int32_t x = lane_i32(L[p].idx, r);
            if (__ballot(lane < cnt && mine == x) != 0) continue;
            if (lane == cnt) mine = x;
            ++cnt;
        }
    }
    if (lane < cnt) a.sel[(int64_t)g * k + lane] = mine;
    if (lane == 0) a.count[g] = cnt;
}

hipError_t launch_select(const SelArgs &a, hipEvent_t *ev, hipStream_t st)
{
    hipLaunchKernelGGL(sel_plan_kernel, dim3(1), dim3(KR_BLOCK), 0, st, a);
    mark(ev, 0, st);
    if (a.max_tiles > 0)
        hipLaunchKernelGGL(sel_tile_kernel, dim3((unsigned)a.max_tiles), dim3(KR_BLOCK), 0, st,
                           a);
    mark(ev, 1, st);
    hipLaunchKernelGGL(sel_final_kernel, dim3(a.n_seg), dim3(KR_BLOCK), 0, st, a);
    return hipGetLastError();
}

}  // namespace kr
