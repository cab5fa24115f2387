// One-comm candidate evaluation and frontier filter, one 256-thread block per slab with
// running-sum tables in LDS (gfx950).
//
// With one comm kernel the candidates of a (partition, frequency) slab are the launch
// positions x SM choices (Section 4.1).  The partition cost model (fluid SM-share
// reading of Sections 3.2 and 4.2; Section 4.3.1 gives no closed form) needs, per
// candidate (p, s), the running sums of time and energy of SM state s + 1 at the launch
// position p and at the kernel j during which the comm kernel ends, those of the
// all-SM state at p and from j to the end, and the raw time and power of kernel j in
// both states.  A block keeps them for one slab in LDS:
//
//   AB  [S + 1][N + 1 + KR_TB_K] {A, B}: A[i] = t[0] + ... + t[i-1] and
//       B[i] = pw[0]*t[0] + ... + pw[i-1]*t[i-1] of each SM state, formed left to right
//       (the running-sum definition, one rounding per addition); state 0 is the all-SM
//       state; rows past N hold A = +inf, so the end-cursor test stops there;
//   TPW [N + 1][S + 1]            {t, pw} in the tables' own row order; row N is a pad,
//       {+inf, 0} for the comm states and zeros for state 0;
//   D0  [N + 2]                   {A0[N] - A0[i], B0[N] - B0[i]}, row N + 1 zeros.
//
// Per slab: the next slab's tables are already in registers (loaded during the previous
// slab) and are stored into TPW; waves 0 and 1 form the A and B columns (one lane per
// column) and the all-SM tails; then every thread evaluates its candidates.  Thread
// (s, r) takes SM choice s and the r-th run of consecutive launch positions.  Its end
// cursor j (largest j with A[j] - A[p] <= Tc) never moves back along the run; each test
// reads the next KR_TB_K rows of its column at once.  The rest of the walk is the
// closed form of the one-comm walk with the pad rows standing in for the case where the
// comm kernel outlasts compute, every line one IEEE fp64 rounding in the cost model's
// order (no FMA contraction), so the results equal the running-sum walk bit for bit.
//
// Filter (GetFrontier, Algorithm 1): per wave and slab, A = least candidate in
// (T, E, index) order and Z = least in (E, T, index) order; every other frontier point
// lies strictly inside their box (T < T_Z, E < E_A).  A, Z and the box members (a few
// per wave) go to the block's unit slot; the merge that follows keeps the exact
// frontier of each partition's units.
#include "kr_filter.h"
#include "kr_launch.h"
#include "kr_wave.h"

namespace kr {

#define KR_TB_THREADS 128  // threads per block (one slab at a time)
#define KR_TB_K 4  // rows per end-cursor test
#define KR_TB_SORT_CAP 1792  // most unit outputs sorted on chip at the block's end (20 B each)
#define KR_TB_OL 96          // filter outputs a block keeps in LDS (more go to device memory)

struct TbLayout {
    int rs;   // records per AB column: N + 1 + KR_TB_K
    int tpw;  // TPW offset (doubles)
    int d0;   // D0 offset (doubles)
    int ol;   // output list offset (doubles): T[KR_TB_OL], E[KR_TB_OL], index[KR_TB_OL]
};

__device__ __forceinline__ TbLayout tb_layout(int N, int S)
{
    TbLayout L;
    L.rs = N + 1 + KR_TB_K;
    L.tpw = 2 * (S + 1) * L.rs;
    L.d0 = L.tpw + 2 * (N + 1) * (S + 1);
    L.ol = L.d0 + 2 * (N + 2);
    return L;
}

typedef double f64x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f64x2 lds2(const double *p) { return *(const f64x2 *)p; }
__device__ __forceinline__ void sts2(double *p, double a, double b)
{
    f64x2 v;
    v.x = a;
    v.y = b;
    *(f64x2 *)p = v;
}

// Register copy of one slab: NE elements per thread of t and pw ([N][S+1] row-major,
// element e = thread + 256 m), and the thread's comm time and power.
template <int NE>
struct TbStage {
    double t[NE], pw[NE];
    double tc, pc;
};

// Least (T, E, index) candidate among those with pred(r) true (fast path when exactly
// one qualifies).  vI[r]: candidate index of slot r.
template <int RR, typename Pred>
__device__ __forceinline__ Key tb_pick(const double (&vT)[RR], const double (&vE)[RR],
                                       const int (&vI)[RR], Pred pred)
{
    int cnt = 0;
    Key one = key_none();
#pragma unroll
    for (int r = 0; r < RR; ++r) {
        const uint64_t m = __ballot(pred(r));
        if (m) {
            cnt += __popcll(m);
            const int L = __ffsll((long long)m) - 1;
            one = Key{lane_u64(dbits(vT[r]), L), lane_u64(dbits(vE[r]), L), lane_i32(vI[r], L)};
        }
    }
    if (cnt == 1) return one;
    Key loc = key_none();
#pragma unroll
    for (int r = 0; r < RR; ++r)
        if (pred(r)) {
            const Key c{dbits(vT[r]), dbits(vE[r]), vI[r]};
            if (kless(c, loc)) loc = c;
        }
    return wave_min_key(loc);
}

// Where a wave's filter outputs go: the block's LDS list (lT, lE, lI, KR_TB_OL entries,
// counter *lcnt), or, when a wave's outputs do not fit there, the unit slot in device
// memory (counter *gcnt).  The one wave whose reservation straddles the list's end
// records its start in *lend: the list's entries from there on are never written.
struct TbOut {
    uint64_t *lT, *lE;
    int32_t *lI;
    int cap;  // list entries in use (KR_TB_OL, less under the test switch)
    int *lcnt, *gcnt, *lend;
    double *oT, *oE;
    int32_t *oI;
};

// A, Z and the box members of the wave's candidates (slots holding +inf are empty).
template <int RR>
__device__ __forceinline__ void tb_filter(const double (&vT)[RR], const double (&vE)[RR],
                                          const int (&vI)[RR], double tl, double el,
                                          const TbOut &ob)
{
    const int lane = threadIdx.x & 63;
    wave_min2_f64(tl, el);
    const uint64_t tab = dbits(tl), ezb = dbits(el);
    if (tab >= KR_INF_BITS) return;
    const Key A = tb_pick<RR>(vT, vE, vI, [&](int r) { return dbits(vT[r]) == tab; });
    Key Z = A;
    int nbox = 0;
    uint32_t rows = 0;
    double TZ = 0.0, EA = bitsd(A.e);
    if (A.e != ezb) {  // else A has the least energy too and dominates everything else
        Z = tb_pick<RR>(vT, vE, vI, [&](int r) { return dbits(vE[r]) == ezb; });
        TZ = bitsd(Z.t);
#pragma unroll
        for (int r = 0; r < RR; ++r) {
            const uint64_t m = __ballot(vT[r] < TZ && vE[r] < EA);
            nbox += __popcll(m);
            rows |= (m != 0 ? 1u : 0u) << r;
        }
    }
    const int nout = (A.e != ezb ? 2 : 1) + nbox;
    int base = 0;
    if (lane == 0) base = atomicAdd(ob.lcnt, nout);
    base = __builtin_amdgcn_readfirstlane(base);
    const bool in_lds = base + nout <= ob.cap;  // uniform
    if (!in_lds) {
        if (lane == 0 && base < ob.cap) *ob.lend = base;
        if (lane == 0) base = atomicAdd(ob.gcnt, nout);
        base = __builtin_amdgcn_readfirstlane(base);
    }
    auto put = [&](int q, uint64_t t, uint64_t e, int32_t i) {
        if (in_lds) {
            ob.lT[q] = t;
            ob.lE[q] = e;
            ob.lI[q] = i;
        } else {
            ob.oT[q] = bitsd(t);
            ob.oE[q] = bitsd(e);
            ob.oI[q] = i;
        }
    };
    if (lane == 0) put(base, A.t, A.e, A.i);
    else if (lane == 1 && A.e != ezb) put(base + 1, Z.t, Z.e, Z.i);
    int at = base + 2;
#pragma unroll
    for (int r = 0; r < RR; ++r)
        if (rows >> r & 1u) {
            const bool b = vT[r] < TZ && vE[r] < EA;
            const uint64_t m = __ballot(b);
            if (b) put(at + lane_rank(m), dbits(vT[r]), dbits(vE[r]), vI[r]);
            at += __popcll(m);
        }
}

// Sort of n keys (T, E, index) in LDS by NT threads: bitonic network whose comparators
// all put the smaller key at the lower index; positions >= n behave as +inf and never
// move, so n need not be a power of two.
template <int NT>
__device__ inline void tb_sort_keys(uint64_t *sT, uint64_t *sE, int32_t *sI, int n)
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
            for (int q = threadIdx.x; q < (m >> 1); q += NT) {
                int lo, hi;
                if (lj == lk - 1) {  // first stage of a merge: mirror within the block
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
            lds_barrier();
        }
    }
}

// Strict prefix-minimum scan of n sorted keys in LDS by NT threads (GetFrontier on the
// sorted order): writes the keys whose E is below every earlier E to o*[0 ..) and
// returns their count (every thread).  sc64, sc32: NT / 64 entries each.
template <int NT>
__device__ inline int tb_frontier_scan(const uint64_t *sT, const uint64_t *sE, const int32_t *sI,
                                       int n, double *oT, double *oE, int32_t *oI,
                                       uint64_t *sc64, int32_t *sc32)
{
    const int per = (n + NT - 1) / NT;
    const int s0 = threadIdx.x * per, s1 = min(n, s0 + per);
    uint64_t m = KR_INF_BITS;
    for (int q = s0; q < s1; ++q) m = MinU64()(m, sE[q]);
    uint64_t tot;
    const uint64_t best0 =
        block_exclusive<uint64_t, MinU64, NT / 64>(m, (uint64_t)KR_INF_BITS, MinU64(), sc64, &tot);
    uint64_t best = best0;
    int nkeep = 0;
    for (int q = s0; q < s1; ++q)
        if (sE[q] < best) {
            ++nkeep;
            best = sE[q];
        }
    int count;
    int opos = block_exclusive<int, SumI32, NT / 64>(nkeep, 0, SumI32(), sc32, &count);
    best = best0;
    for (int q = s0; q < s1; ++q) {
        const uint64_t e = sE[q];
        if (e < best) {
            oT[opos] = bitsd(sT[q]);
            oE[opos] = bitsd(e);
            oI[opos] = sI[q];
            ++opos;
            best = e;
        }
    }
    return count;
}

// Block (p, b): partition p, frequencies [b*fb, min(F, (b+1)*fb)), NT = 128 threads.
// SC = S (SM choices), NE = elements per thread of a slab copy, SPAN = positions per run.
// The tq walk positions (all positions, or all but the last when n_pos = N + 1) form 8
// runs of SPAN; positions past tq - 1 are walked as position tq - 1 (so the cursors stay
// in range) and dropped before the filter, so every candidate enters the filter once and
// a unit never outputs more points than its slot holds.  Thread (s, g) evaluates two runs of SM choice s, runs g
// and g + 4, one position of each per round, so every round carries two independent
// walks.  With n_pos = N + 1 the last position launches the comm kernel after the last
// compute kernel: T = A0[N] + Tc and E = (p_static T + B0[N]) + pc Tc (the walk's
// operations with nothing but zeros added), taken by the threads of g = 3.
//
// The rounds are software-pipelined: round k + 1's launch-position records are read
// before round k's arithmetic and its end cursor is settled after it, so LDS latency
// overlaps the fp64 chains of the round before.
template <int NT, int SC, int NE, int SPAN>
__global__ void __launch_bounds__(NT, 2) eval_table_kernel(EvalArgs a, UnitOut o)
{
    constexpr int S = SC, S1 = SC + 1, RT = 2 * SPAN + 1;  // slots: two runs + closed form
    static_assert(NT == 4 * SC, "four thread groups of one SM choice each");
    // 16-byte aligned: the {A, B} and {t, pw} records are read as 16-byte pairs
    extern __shared__ __attribute__((aligned(16))) double lds[];
    __shared__ int s_cnt, s_gcnt, s_lend;
    __shared__ uint64_t s_sc64[NT / 64];
    __shared__ int32_t s_sc32[NT / 64];
    const int N = a.N;
    const TbLayout lay = tb_layout(N, S);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int p = blockIdx.x / a.nfb, fbk = blockIdx.x - p * a.nfb;
    const int f0 = fbk * a.fb, f1 = min(a.F, f0 + a.fb);
    const int slab = N * S1;
    double *const AB = lds, *const TPW = lds + lay.tpw, *const D0 = lds + lay.d0;

    // pad rows (never overwritten): A = +inf past row N of every column, the raw row N,
    // and the zero tail row N + 1
    for (int x = tid; x < S1 * KR_TB_K; x += NT) {
        const int c = x / KR_TB_K, i = N + 1 + x % KR_TB_K;
        sts2(AB + 2 * (c * lay.rs + i), INFINITY, 0.0);
    }
    for (int c = tid; c < S1; c += NT) {
        sts2(TPW + 2 * (N * S1 + c), c == 0 ? 0.0 : INFINITY, 0.0);
        sts2(AB + 2 * (c * lay.rs), 0.0, 0.0);
    }
    if (tid == 0) {
        sts2(D0 + 2 * (N + 1), 0.0, 0.0);
        s_cnt = 0;
        s_gcnt = 0;
        s_lend = a.tb_ol;
    }

    const int s = tid % S, g = tid / S;
    const int tq = a.tq;                     // walk positions 0 .. tq - 1
    const bool closed = a.tclosed && g == 3;  // this thread also takes position N
    const int pa0 = g * SPAN, pb0 = (g + 4) * SPAN;
    // candidate index of each slot, less f * Cf
    int posS[RT];
#pragma unroll
    for (int k = 0; k < SPAN; ++k) {
        posS[k] = min(pa0 + k, tq - 1) * S + s;
        posS[SPAN + k] = min(pb0 + k, tq - 1) * S + s;
    }
    posS[RT - 1] = N * S + s;

    TbStage<NE> st;
    auto load_stage = [&](int f) {
        const size_t pf = (size_t)p * a.F + f;
        const double *gt = a.t + pf * slab, *gp = a.pw + pf * slab;
#pragma unroll
        for (int m = 0; m < NE; ++m) {  // unsigned 32-bit offsets from a uniform base
            const uint32_t ec = min((uint32_t)(tid + NT * m), (uint32_t)(slab - 1));
            st.t[m] = gt[ec];
            st.pw[m] = gp[ec];
        }
        st.tc = a.tc[pf * S + s];
        st.pc = a.pc[pf * S + s];
    };
    load_stage(f0);

    const size_t slot0 = (size_t)p * a.C + (size_t)f0 * a.Cf;
    double *const oT = o.T + slot0, *const oE = o.E + slot0;
    int32_t *const oI = o.I + slot0;
    TbOut ob;
    ob.lT = (uint64_t *)(lds + lay.ol);
    ob.lE = ob.lT + KR_TB_OL;
    ob.lI = (int32_t *)(ob.lE + KR_TB_OL);
    ob.cap = a.tb_ol;
    ob.lcnt = &s_cnt;
    ob.gcnt = &s_gcnt;
    ob.lend = &s_lend;
    ob.oT = oT;
    ob.oE = oE;
    ob.oI = oI;
    const double p_static = a.p_static;
    // this thread's column (state s + 1) and the all-SM column 0
    const double *const abs_ = AB + 2 * (s + 1) * lay.rs, *const ab0 = AB;

    for (int f = f0; f < f1; ++f) {
        lds_barrier();  // every read of the previous slab's tables is done
#pragma unroll
        for (int m = 0; m < NE; ++m) {
            const int e = tid + NT * m;
            if (e < slab) sts2(TPW + 2 * e, st.t[m], st.pw[m]);
        }
        const double Tc = st.tc, ctail = st.pc * st.tc;
        if (f + 1 < f1) load_stage(f + 1);
        lds_barrier();  // TPW holds slab f (the next slab's loads stay in flight)

        // Running sums, one lane per state: wave 0 the times, wave 1 the energies; then
        // the same waves form the all-SM tails from the totals.
        if (lane < S1) {
            const double *src = TPW + 2 * lane;
            double *col = AB + 2 * lane * lay.rs + wave;  // A or B half of the records
            double acc = 0.0;
            int i0 = 0;
            for (; i0 + 16 <= N; i0 += 16) {
                f64x2 v[16];
#pragma unroll
                for (int q = 0; q < 16; ++q) v[q] = lds2(src + 2 * S1 * (i0 + q));
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    acc = acc + (wave == 0 ? v[q].x : v[q].y * v[q].x);
                    col[2 * (i0 + q + 1)] = acc;
                }
            }
            for (; i0 < N; ++i0) {
                const f64x2 v = lds2(src + 2 * S1 * i0);
                acc = acc + (wave == 0 ? v.x : v.y * v.x);
                col[2 * (i0 + 1)] = acc;
            }
        }
        {
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
            const double *z = ab0 + wave;  // all-SM column, A or B half
            const double tot = z[2 * N];
            for (int i = lane; i <= N; i += 64) D0[2 * i + wave] = tot - z[2 * i];
        }
        lds_barrier();  // AB and D0 hold slab f

        // Evaluation: two walks per round, software-pipelined over the rounds.
        double vT[RT], vE[RT];
        double tl = INFINITY, el = INFINITY;
        f64x2 abp[2], z0p[2];                        // records at the launch positions
        f64x2 abj[2], tpj[2], t0j[2], d0[2], d1[2];  // records at the end kernels j
        int j[2];
        // end cursors of both walks from st[w]: largest j with A[j] - A[p] <= Tc
        auto settle = [&](int st0, int st1) {
            int jj[2] = {st0, st1};
            bool go[2] = {true, true};
            do {
#pragma unroll
                for (int w = 0; w < 2; ++w)
                    if (go[w]) {
                        const double *q = abs_ + 2 * jj[w];
                        const double a1 = q[2], a2 = q[4], a3 = q[6], a4 = q[8], ap = abp[w].x;
                        const int d = (a1 - ap <= Tc ? 1 : 0) + (a2 - ap <= Tc ? 1 : 0) +
                                      (a3 - ap <= Tc ? 1 : 0) + (a4 - ap <= Tc ? 1 : 0);
                        jj[w] += d;
                        go[w] = d == KR_TB_K;
                    }
            } while (__ballot(go[0] || go[1]));
            j[0] = jj[0];
            j[1] = jj[1];
        };
        auto fetch_j = [&](int w) {
            abj[w] = lds2(abs_ + 2 * j[w]);
            tpj[w] = lds2(TPW + 2 * (j[w] * S1 + s + 1));
            t0j[w] = lds2(TPW + 2 * (j[w] * S1));
            d0[w] = lds2(D0 + 2 * j[w]);
            d1[w] = lds2(D0 + 2 * j[w] + 2);
        };
        {
            const int qa = min(pa0, tq - 1), qb = min(pb0, tq - 1);
            abp[0] = lds2(abs_ + 2 * qa);
            z0p[0] = lds2(ab0 + 2 * qa);
            abp[1] = lds2(abs_ + 2 * qb);
            z0p[1] = lds2(ab0 + 2 * qb);
            settle(qa, qb);
            fetch_j(0);
            fetch_j(1);
        }
#pragma unroll
        for (int k = 0; k < SPAN; ++k) {
            // this round's inputs, then the next round's launch-position records
            f64x2 cabp[2], cz0p[2], cabj[2], ctpj[2], ct0j[2], cd0[2], cd1[2];
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                cabp[w] = abp[w];
                cz0p[w] = z0p[w];
                cabj[w] = abj[w];
                ctpj[w] = tpj[w];
                ct0j[w] = t0j[w];
                cd0[w] = d0[w];
                cd1[w] = d1[w];
            }
            const bool more = k + 1 < SPAN;  // folded by the unrolling
            const int pn[2] = {min(pa0 + k + 1, tq - 1), min(pb0 + k + 1, tq - 1)};
            if (more) {
#pragma unroll
                for (int w = 0; w < 2; ++w) {
                    abp[w] = lds2(abs_ + 2 * pn[w]);
                    z0p[w] = lds2(ab0 + 2 * pn[w]);
                }
            }
            // round k of both walks: the rest of the walk (the comm phase ends inside
            // kernel j, or compute ends first: then row j = N is the pad and nothing
            // more is added)
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                const double rem = Tc - (cabj[w].x - cabp[w].x);
                double Ec = cz0p[w].y + (cabj[w].y - cabp[w].y);
                Ec = Ec + ctpj[w].y * rem;
                const double wf = __builtin_fmax(1.0 - rem / ctpj[w].x, 0.0);
                const bool part = wf < 1.0;
                const double need = wf * ct0j[w].x;
                const double used = part ? need : 0.0;
                Ec = Ec + ct0j[w].y * used;
                Ec = Ec + (part ? cd1[w].y : cd0[w].y);
                const double el_ = used + (part ? cd1[w].x : cd0[w].x);
                const double T = (cz0p[w].x + Tc) + el_;
                double E = p_static * T;
                E = E + Ec;
                E = E + ctail;
                vT[w * SPAN + k] = T;
                vE[w * SPAN + k] = E;
                tl = vmin(tl, T);
                el = vmin(el, E);
            }
            if (more) {
                settle(max(pn[0], j[0]), max(pn[1], j[1]));
                fetch_j(0);
                fetch_j(1);
            }
        }
        {  // position N, comm launched after the last compute kernel
            const f64x2 zN = lds2(ab0 + 2 * N);
            const double T = zN.x + Tc;
            double E = p_static * T;
            E = E + zN.y;
            E = E + ctail;
            vT[RT - 1] = closed ? T : INFINITY;
            vE[RT - 1] = closed ? E : INFINITY;
            tl = vmin(tl, vT[RT - 1]);
            el = vmin(el, vE[RT - 1]);
        }
        if (8 * SPAN > tq) {  // uniform: some runs repeat position tq - 1; keep one copy
#pragma unroll
            for (int k = 0; k < SPAN; ++k) {
                if (pa0 + k >= tq) vT[k] = vE[k] = INFINITY;
                if (pb0 + k >= tq) vT[SPAN + k] = vE[SPAN + k] = INFINITY;
            }
        }
        int vI[RT];
        const int fC = f * a.Cf;
#pragma unroll
        for (int r = 0; r < RT; ++r) vI[r] = fC + posS[r];
        tb_filter<RT>(vT, vE, vI, tl, el, ob);
    }
    // The unit's exact frontier: its outputs (a few per wave and slab, in the LDS list)
    // are sorted there and the strict prefix-minimum scan (GetFrontier) writes the kept
    // points to the unit slot, so the merge that follows sees one short staircase per
    // unit.  When some outputs went to device memory, the list joins them there and all
    // are sorted in the LDS of the tables, which are dead now; a unit with more outputs
    // than that holds is left unsorted (the merge keeps the same frontier either way).
    __syncthreads();
    const int nl = min(s_cnt, s_lend), ng = s_gcnt;  // every output once: ng + nl <= slot
    if (ng == 0) {
        tb_sort_keys<NT>(ob.lT, ob.lE, ob.lI, nl);
        const int kept = tb_frontier_scan<NT>(ob.lT, ob.lE, ob.lI, nl, oT, oE, oI, s_sc64, s_sc32);
        if (tid == 0) o.cnt[blockIdx.x] = kept;
        return;
    }
    for (int x = tid; x < nl; x += NT) {
        oT[ng + x] = bitsd(ob.lT[x]);
        oE[ng + x] = bitsd(ob.lE[x]);
        oI[ng + x] = ob.lI[x];
    }
    __syncthreads();
    const int n = ng + nl;
    // sort area: 20 bytes per output within the block's table LDS
    const int cap = min(KR_TB_SORT_CAP, lay.ol * 8 / 20);
    if (n <= cap) {
        uint64_t *sT = (uint64_t *)lds, *sE = sT + cap;
        int32_t *sI = (int32_t *)(sE + cap);
        // the block's own stores, ordered by the barrier above: plain loads (the CU's
        // cache holds no line of this slot from before, and its stores write through to
        // the L2 these loads read)
        for (int x = tid; x < n; x += NT) {
            sT[x] = dbits(oT[x]);
            sE[x] = dbits(oE[x]);
            sI[x] = oI[x];
        }
        __syncthreads();
        tb_sort_keys<NT>(sT, sE, sI, n);
        const int kept = tb_frontier_scan<NT>(sT, sE, sI, n, oT, oE, oI, s_sc64, s_sc32);
        if (tid == 0) o.cnt[blockIdx.x] = kept;
    } else if (tid == 0) {
        o.cnt[blockIdx.x] = n;
    }
}

template <int NT, int NE, int SPAN>
static void launch_tb(const EvalArgs &a, const UnitOut &o, size_t lds, hipStream_t st)
{
    hipLaunchKernelGGL((eval_table_kernel<NT, 32, NE, SPAN>), dim3(a.P * a.nfb), dim3(NT), lds,
                       st, a, o);
}

hipError_t launch_eval_filter_table(const EvalArgs &a, const UnitOut &o, hipStream_t st)
{
    const size_t lds = (size_t)a.lds_doubles * sizeof(double);
    constexpr int NT = KR_TB_THREADS;
    if (a.S != 32 || (a.N * 33 + NT - 1) / NT > 9) return hipErrorInvalidValue;
    switch (a.span) {  // walk positions per run
    case 1: launch_tb<NT, 9, 1>(a, o, lds, st); break;
    case 2: launch_tb<NT, 9, 2>(a, o, lds, st); break;
    case 3: launch_tb<NT, 9, 3>(a, o, lds, st); break;
    case 4: launch_tb<NT, 9, 4>(a, o, lds, st); break;
    case 5: launch_tb<NT, 9, 5>(a, o, lds, st); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace kr
