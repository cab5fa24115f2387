// C ABI of libkareus_mi355x.so: argument checks, workspace layout and launch order.
// Declarations and contracts: include/kareus.h.
#include <algorithm>
#include <cstdlib>
#include <cstring>

#include "../../include/kareus.h"
#include "kr_filter.h"
#include "kr_launch.h"

using namespace kr;

namespace {

constexpr size_t kLdsBudget = 65536;
constexpr size_t kLdsPerCu = 160 * 1024;
constexpr int kSurvDoubles = KR_SURV_CAP * 20 / 8;
constexpr size_t kAlign = 256;
constexpr int64_t kWaveBlocksPerSlot = 32;

// Bump allocator over the caller's workspace (or a size query when base == nullptr).
struct Carve {
    char *base;
    size_t used = 0;
    explicit Carve(void *b) : base((char *)b) {}
    template <typename T>
    T *take(size_t n)
    {
        used = (used + kAlign - 1) / kAlign * kAlign;
        T *p = base ? (T *)(base + used) : nullptr;
        used += n * sizeof(T);
        return p;
    }
};

bool space_ok(const kr_space *s)
{
    return s && s->n_parts >= 1 && s->n_kernels >= 1 && (s->n_comm == 1 || s->n_comm == 2) &&
           s->n_freq >= 1 && s->n_sm >= 1 && s->n_pos >= 1 && s->n_pos <= s->n_kernels + 1 &&
           s->n_pos <= 0x7FFF && s->p_static >= 0.0;
}

int64_t cand_per_freq(const kr_space *s)
{
    const int64_t S = s->n_sm;
    if (s->n_comm == 1) return (int64_t)s->n_pos * S;
    const int64_t npp = (int64_t)s->n_pos * (s->n_pos + 1) / 2;
    return npp * S * S;
}

// One comm kernel and at most 64 SM choices: one wave per slab.  Lane (h, s) takes SM
// choice s and the h-th run of launch positions, R of them per register chunk.
bool wave_plan(EvalArgs *a)
{
    if (a->M != 1 || a->S > 64) return false;
    const int64_t rows = (int64_t)(a->N + KR_PAD) * (a->S + 1);  // slab and pad rows
    const int64_t rows16 = (rows + 1) / 2 * 2;  // keeps the second table 16-byte aligned
    const int64_t lds = 2 * rows16 + 2 * (a->N + 2);  // t, pw, all-SM column sums
    if ((size_t)lds * 8 > kLdsBudget) return false;
    a->wave = 1;
    a->w_pw = (int)rows16;
    a->w_a0 = (int)(2 * rows16);
    a->lds_doubles = (int)lds;
    // runs of span positions, a multiple of 8 when there are several (the running-sum
    // pass keeps a lane's starting sums at 8-row block boundaries); the last run takes
    // the rest
    a->H = 64 / a->S;
    a->span = a->H == 1 ? a->n_pos : std::max(8, a->n_pos / a->H / 8 * 8);
    const int last = std::max(0, a->n_pos - (a->H - 1) * a->span);
    const int maxrun = std::max(std::min(a->span, a->n_pos), last);
    a->R = maxrun <= 2 ? 2 : maxrun <= 4 ? 4 : maxrun <= 8 ? 8 : 17;
    a->nch = (maxrun + a->R - 1) / a->R;
    a->fixed32 = a->N == 32 && a->S == 32 && a->n_pos == 33 && a->H == 2 && a->span == 16 &&
                 a->R == 17 && a->nch == 1 && std::min(a->span, last) >= a->R - 1 &&
                 a->w_pw == KR_FIX32_PW && a->w_a0 == 2 * KR_FIX32_PW;
    // filter scratch: the pad rows of each table
    // (the power pad holds cap doubles of E, then cap ints of indices)
    a->wcap = (int)std::min<int64_t>(64, KR_PAD * (a->S + 1) * 2 / 3);
    // a few times more one-wave blocks than fit on the chip at once, so the
    // dispatcher balances uneven slabs; within a block slab copies overlap the filter
    const int64_t resident = std::max<int64_t>(1, std::min<int64_t>(16, kLdsPerCu / (lds * 8)));
    const int64_t target = kWaveBlocksPerSlot * 256 * resident;
    int64_t nfb = std::max<int64_t>(1, (target + a->P - 1) / a->P);
    nfb = std::min<int64_t>(nfb, a->F);
    a->fb = (int)((a->F + nfb - 1) / nfb);
    a->nfb = (a->F + a->fb - 1) / a->fb;
    return true;
}

// Two comm kernels and at most 8 SM choices: one wave per slab, lane (s1, s2).
bool pair_plan(EvalArgs *a)
{
    if (a->M != 2 || a->S > 8) return false;
    const int64_t S1 = a->S + 1;
    const int64_t slab16 = ((int64_t)a->N * S1 + 1) / 2 * 2;
    a->q_pw = (int)slab16;
    a->q_ab = (int)(2 * slab16);
    a->q_f = (int)(a->q_ab + 2 * (a->N + 1) * S1);  // {A, B} records
    a->q_c = (int)(a->q_f + 6 * (int64_t)a->n_pos * a->S);  // 6-double records
    constexpr int NW = KR_PAIR_WAVES;
    a->q_sc = a->q_c + NW * 6 * 64;                     // one set per wave
    const int64_t lds = a->q_sc + NW * (64 + 64 + 32);  // scratch T, E, indices per wave
    if ((size_t)lds * 8 > kLdsBudget) return false;
    a->pair = 1;
    a->lds_doubles = (int)lds;
    // each wave's slab-end reduction sorts in its share of the second-phase tables (20
    // bytes per point); a test-only switch lowers the cap (0: never), so tests reach the
    // unreduced path
    a->pair_scap = (a->q_sc - a->q_f) / NW * 8 / 20;
    if (const char *e = std::getenv("KR_TEST_PAIR_SORT_CAP"))
        a->pair_scap = std::max(0, std::min(a->pair_scap, std::atoi(e)));
    // a slab is tens of thousands of candidates: one block per slab unless there are too
    // few slabs to fill the chip many times over (short tails)
    const int64_t resident = std::max<int64_t>(1, std::min<int64_t>(16, kLdsPerCu / (lds * 8)));
    const int64_t target = 8 * 256 * resident;
    int64_t nfb = std::max<int64_t>(1, (target + a->P - 1) / a->P);
    nfb = std::min<int64_t>(nfb, a->F);
    a->fb = (int)((a->F + nfb - 1) / nfb);
    a->nfb = (a->F + a->fb - 1) / a->fb;
    // NW units per block, one per wave with the launch positions it owns: a unit's slot
    // holds every candidate the largest share has in fb slabs
    int64_t share[NW] = {};
    for (int p1 = 0; p1 < a->n_pos; ++p1) share[pair_owner_host(p1, NW)] += a->n_pos - p1;
    a->uper = NW * (int64_t)a->nfb;
    a->ustride = (int64_t)a->fb * *std::max_element(share, share + NW) * a->S * a->S;
    a->useg = a->uper * a->ustride;
    return true;
}

// Shape of the evaluation launch; false if the slab does not fit on chip.
bool eval_plan(const kr_space *s, bool fused, EvalArgs *a)
{
    std::memset(a, 0, sizeof(*a));
    a->P = s->n_parts;
    a->N = s->n_kernels;
    a->M = s->n_comm;
    a->F = s->n_freq;
    a->S = s->n_sm;
    a->n_pos = s->n_pos;
    a->n_pp = s->n_pos * (s->n_pos + 1) / 2;
    const int64_t cf = cand_per_freq(s);
    if (cf > 0x7FFFFFFF / s->n_freq) return false;
    a->Cf = (int)cf;
    a->C = cf * s->n_freq;
    a->p_static = s->p_static;
    const int64_t S1 = a->S + 1;
    if (fused && wave_plan(a)) {
        a->useg = a->C;
        a->uper = a->nfb;
        a->ustride = (int64_t)a->fb * a->Cf;
        return true;
    }
    if (fused && pair_plan(a)) return true;
    const int64_t staged = 2 * a->N * S1 + 2 * a->M * a->S;  // t, pw, tc, pc
    const int64_t sums = 2 * (a->N + 1) * S1;
    const int64_t pairs = a->M == 2 ? (a->n_pp * 4 + 7) / 8 : 0;
    a->surv_off = (int)(staged + sums + pairs);
    a->lds_doubles = a->surv_off + (fused ? kSurvDoubles : 0);
    if ((size_t)a->lds_doubles * 8 > kLdsBudget) return false;
    if (!fused) return true;
    // register prefetch: pf doubles per thread of each table, one of the comm tables
    const int64_t slab = a->N * S1;
    a->pf = (int)((slab + KR_BLOCK - 1) / KR_BLOCK);
    if (a->pf > 8 || a->M * a->S > KR_BLOCK) return false;
    a->one_comm = a->M == 1 && a->S <= KR_BLOCK;
    if (a->one_comm) {
        a->nchunk = KR_BLOCK / a->S;
        a->cpt = (int)std::min<int64_t>(8, (a->n_pos + a->nchunk - 1) / a->nchunk);
        a->ntiles = (a->n_pos + a->nchunk * a->cpt - 1) / (a->nchunk * a->cpt);
        a->tile = a->nchunk * a->cpt * a->S;
        // one tile per slab: the staged time table is dead once the tile is evaluated,
        // so the survivor list can live on top of it
        if (a->ntiles == 1 && a->N * S1 >= kSurvDoubles) {
            a->surv_off = 0;
            a->lds_doubles -= kSurvDoubles;
        }
    } else {
        a->cpt = (int)std::min<int64_t>(8, (a->Cf + KR_BLOCK - 1) / KR_BLOCK);
        a->tile = KR_BLOCK * a->cpt;
        a->ntiles = (a->Cf + a->tile - 1) / a->tile;
    }
    // enough blocks to fill every CU at the LDS-limited occupancy
    const size_t per_block = (size_t)a->lds_doubles * 8 + 1024;
    const int64_t resident = std::max<int64_t>(1, std::min<size_t>(8, kLdsPerCu / per_block));
    const int64_t target = 256 * resident;
    int64_t nfb = std::max<int64_t>(1, (target + a->P - 1) / a->P);
    nfb = std::min<int64_t>(nfb, a->F);
    a->fb = (int)((a->F + nfb - 1) / nfb);
    a->nfb = (a->F + a->fb - 1) / a->fb;
    a->useg = a->C;
    a->uper = a->nfb;
    a->ustride = (int64_t)a->fb * a->Cf;
    return true;
}

// The input check of the cost tables, when the caller asks for a status word.
hipError_t check_tables(const kr_space *s, const double *t, const double *pw, const double *tc,
                        const double *pc, int32_t *status, hipStream_t st)
{
    const int64_t slabs = (int64_t)s->n_parts * s->n_freq;
    const int64_t nt = slabs * s->n_kernels * (s->n_sm + 1), nc = slabs * s->n_comm * s->n_sm;
    const double *xs[4] = {t, pw, tc, pc};
    const int64_t n[4] = {nt, nt, nc, nc};
    return launch_check(xs, n, 4, status, st);
}

// Caller-owned events recorded around a phase (kr_set_phase_events), one setting per
// host thread: a call reads only its own thread's entries, so threads never race on them.
thread_local hipEvent_t g_phase_ev[6][2] = {};

void phase_mark(int phase, int which, hipStream_t st)
{
    if (g_phase_ev[phase][0] && g_phase_ev[phase][1])
        (void)hipEventRecord(g_phase_ev[phase][which], st);
}

struct FilterWs {
    int64_t *seg_off, *unit_base;
    int32_t *ucnt, *fcnt, *runcnt, *lists;
    PointBufs buf[2];
    uint8_t *flags;
};

FilterWs carve_filter(Carve &c, int64_t n_total, int n_seg, int64_t n_units, bool own_seg_off)
{
    FilterWs w;
    const int64_t n = std::max<int64_t>(n_total, 1);
    w.seg_off = own_seg_off ? c.take<int64_t>(n_seg + 1) : nullptr;
    w.unit_base = c.take<int64_t>(n_seg + 1);
    w.ucnt = c.take<int32_t>(std::max<int64_t>(n_units, 1));
    w.fcnt = c.take<int32_t>(std::max(n_seg, 1));
    w.runcnt = c.take<int32_t>(n_total / KR_FIN_CAP + n_seg + 1);
    w.lists = c.take<int32_t>(2 * (int64_t)n_seg + 2);
    for (int i = 0; i < 2; ++i) {
        w.buf[i].T = c.take<double>(n);
        w.buf[i].E = c.take<double>(n);
        w.buf[i].I = c.take<int32_t>(n);
    }
    w.flags = c.take<uint8_t>((n + 3) / 4 * 4);
    return w;
}

// Union of every segment's unit frontiers, then the CSR output.
kr_status finish_segments(const SegLayout &L, FilterWs &w, int64_t cap, int64_t *out_off,
                          int32_t *out_idx, double *out_T, double *out_E, hipStream_t st)
{
    phase_mark(KR_PHASE_MERGE, 0, st);
    if (launch_finalize(L, w.buf[0], w.ucnt, w.buf[1], w.fcnt, w.runcnt, w.flags, w.lists, st) !=
        hipSuccess)
        return KR_EHIP;
    if (launch_output(L, w.buf[1], w.fcnt, cap, out_off, out_idx, out_T, out_E, st) != hipSuccess)
        return KR_EHIP;
    phase_mark(KR_PHASE_MERGE, 1, st);
    return KR_OK;
}

}  // namespace

extern "C" {

int64_t kr_candidates_per_partition(const kr_space *space)
{
    if (!space_ok(space)) return 0;
    return cand_per_freq(space) * space->n_freq;
}

kr_status kr_evaluate_partition(const kr_space *space, const double *t, const double *pw,
                                const double *tc, const double *pc, double *T_out, double *E_out,
                                int32_t *status_out, void *stream)
{
    if (!space_ok(space) || !t || !pw || !tc || !pc || !T_out || !E_out) return KR_EINVAL;
    EvalArgs a;
    if (!eval_plan(space, false, &a)) return KR_EUNSUPPORTED;
    a.t = t;
    a.pw = pw;
    a.tc = tc;
    a.pc = pc;
    a.T_out = T_out;
    a.E_out = E_out;
    if (status_out && check_tables(space, t, pw, tc, pc, status_out, (hipStream_t)stream) != hipSuccess)
        return KR_EHIP;
    return launch_eval(a, (hipStream_t)stream) == hipSuccess ? KR_OK : KR_EHIP;
}

size_t kr_pareto_filter_workspace(int64_t n_total, int32_t n_seg)
{
    if (n_total < 0 || n_seg < 0) return 0;
    const int64_t n_units = (n_total + KR_TILE - 1) / KR_TILE + n_seg;
    Carve c(nullptr);
    carve_filter(c, n_total, n_seg, n_units, false);
    return c.used;
}

kr_status kr_pareto_filter(int64_t n_total, const double *T, const double *E,
                           const int64_t *seg_off, int32_t n_seg, int64_t cap, int64_t *out_off,
                           int32_t *out_idx, double *out_T, double *out_E, int32_t *status_out,
                           void *ws, size_t ws_bytes, void *stream)
{
    if (n_total < 0 || n_seg < 0 || cap < 0 || !seg_off || !out_off ||
        (n_total > 0 && (!T || !E)) || (cap > 0 && (!out_idx || !out_T || !out_E)) || !ws)
        return KR_EINVAL;
    if (ws_bytes < kr_pareto_filter_workspace(n_total, n_seg)) return KR_ECAPACITY;
    hipStream_t st = (hipStream_t)stream;
    const int64_t n_units = (n_total + KR_TILE - 1) / KR_TILE + n_seg;
    if (status_out) {
        const double *xs[2] = {T, E};
        const int64_t n[2] = {n_total, n_total};
        if (launch_check(xs, n, 2, status_out, st) != hipSuccess) return KR_EHIP;
    }
    Carve c(ws);
    FilterWs w = carve_filter(c, n_total, n_seg, n_units, false);
    SegLayout L;
    L.seg_off = seg_off;
    L.unit_base = w.unit_base;
    L.n_seg = n_seg;
    L.unit_stride = KR_TILE;
    if (n_seg > 0 &&
        launch_tile_layout(seg_off, w.unit_base, n_seg, KR_TILE, w.lists, st) != hipSuccess)
        return KR_EHIP;
    UnitOut o{w.buf[0].T, w.buf[0].E, w.buf[0].I, w.ucnt};
    if (n_seg > 0 && launch_pareto_tiles(T, E, L, n_units, o, st) != hipSuccess) return KR_EHIP;
    return finish_segments(L, w, cap, out_off, out_idx, out_T, out_E, st);
}

size_t kr_evaluate_and_filter_workspace(const kr_space *space)
{
    EvalArgs a;
    if (!space_ok(space) || !eval_plan(space, true, &a)) return 0;
    Carve c(nullptr);
    carve_filter(c, (int64_t)a.P * a.useg, a.P, (int64_t)a.P * a.uper, true);
    return c.used;
}

kr_status kr_evaluate_and_filter(const kr_space *space, const double *t, const double *pw,
                                 const double *tc, const double *pc, int64_t cap, int64_t *out_off,
                                 int32_t *out_idx, double *out_T, double *out_E,
                                 int32_t *status_out, void *ws, size_t ws_bytes, void *stream)
{
    if (!space_ok(space) || !t || !pw || !tc || !pc || cap < 0 || !out_off ||
        (cap > 0 && (!out_idx || !out_T || !out_E)) || !ws)
        return KR_EINVAL;
    EvalArgs a;
    if (!eval_plan(space, true, &a)) return KR_EUNSUPPORTED;
    const size_t need = kr_evaluate_and_filter_workspace(space);
    if (need == 0 || ws_bytes < need) return KR_ECAPACITY;
    hipStream_t st = (hipStream_t)stream;
    a.t = t;
    a.pw = pw;
    a.tc = tc;
    a.pc = pc;
    Carve c(ws);
    FilterWs w = carve_filter(c, (int64_t)a.P * a.useg, a.P, (int64_t)a.P * a.uper, true);
    if (launch_uniform_layout(w.seg_off, w.unit_base, a.P, a.useg, a.uper, w.lists, st) !=
        hipSuccess)
        return KR_EHIP;
    UnitOut o{w.buf[0].T, w.buf[0].E, w.buf[0].I, w.ucnt};
    a.dma16 = (a.wave || a.pair) && (a.N * (a.S + 1)) % 2 == 0 && (uintptr_t)t % 16 == 0 &&
              (uintptr_t)pw % 16 == 0;
    if (status_out && check_tables(space, t, pw, tc, pc, status_out, st) != hipSuccess)
        return KR_EHIP;
    phase_mark(KR_PHASE_EVAL_TILE, 0, st);
    const hipError_t le = a.wave   ? launch_eval_filter_wave(a, o, st)
                          : a.pair ? launch_eval_filter_pair(a, o, st)
                                   : launch_eval_filter(a, o, st);
    if (le != hipSuccess) return KR_EHIP;
    phase_mark(KR_PHASE_EVAL_TILE, 1, st);
    SegLayout L;
    L.seg_off = w.seg_off;
    L.unit_base = w.unit_base;
    L.n_seg = a.P;
    L.unit_stride = a.ustride;
    return finish_segments(L, w, cap, out_off, out_idx, out_T, out_E, st);
}

size_t kr_compose_frontiers_workspace(int32_t n_parts, int32_t n_bins)
{
    if (n_parts < 1 || n_bins < 2) return 0;
    const size_t P = n_parts, B = n_bins;
    Carve c(nullptr);
    c.take<double>(P);
    c.take<double>(P);
    c.take<int64_t>(P);
    c.take<int64_t>(P);
    c.take<int64_t>(P + 1);
    c.take<int64_t>(1);
    c.take<uint64_t>(B + 8 * P);
    c.take<int32_t>(B + 8 * P);
    c.take<int32_t>(B + 8 * P);
    c.take<int32_t>(B + 8 * P);
    c.take<double>(B + 8 * P);
    c.take<int32_t>(P);
    c.take<double>(P * B);
    c.take<int32_t>(1);
    c.take<double>((B + KR_ST_CHUNK - 1) / KR_ST_CHUNK);
    c.take<int32_t>((B + KR_ST_CHUNK - 1) / KR_ST_CHUNK);
    return c.used;
}

kr_status kr_compose_frontiers(int32_t n_parts, const int64_t *off, const double *T,
                               const double *E, int32_t n_bins, double delta, double *F_out,
                               int32_t *bp_out, int32_t *bp_off_out, int32_t *pt_bin_out,
                               double *info_out,
                               int32_t *L_out, int32_t *stair_bin, double *stair_Tlo,
                               double *stair_E, int32_t *n_stair, int32_t *status_out, void *ws,
                               size_t ws_bytes, void *stream)
{
    if (n_parts < 1 || n_bins < 2 || !off || !T || !E || !F_out || !bp_out || !pt_bin_out ||
        !info_out || !L_out || !stair_bin || !stair_Tlo || !stair_E || !n_stair || !status_out ||
        !ws || !(delta >= 0.0))
        return KR_EINVAL;
    if (ws_bytes < kr_compose_frontiers_workspace(n_parts, n_bins)) return KR_ECAPACITY;
    const size_t P = n_parts, B = n_bins;
    Carve c(ws);
    ComposeWs w;
    w.tmin = c.take<double>(P);
    w.range = c.take<double>(P);
    w.Mk = c.take<int64_t>(P);
    w.Lk = c.take<int64_t>(P);
    w.eoff = c.take<int64_t>(P + 1);
    w.mmax = c.take<int64_t>(1);
    w.ebits = c.take<uint64_t>(B + 8 * P);
    w.earg = c.take<int32_t>(B + 8 * P);
    w.ob2 = c.take<int32_t>(B + 8 * P);
    w.oarg = c.take<int32_t>(B + 8 * P);
    w.oe = c.take<double>(B + 8 * P);
    w.occ = c.take<int32_t>(P);
    w.Fh = c.take<double>(P * B);
    w.ticket = c.take<int32_t>(1);
    w.chmin = c.take<double>((B + KR_ST_CHUNK - 1) / KR_ST_CHUNK);
    w.chcnt = c.take<int32_t>((B + KR_ST_CHUNK - 1) / KR_ST_CHUNK);
    ComposeArgs a;
    a.P = n_parts;
    a.B = n_bins;
    a.delta_in = delta;
    a.off = off;
    a.T = T;
    a.E = E;
    a.F_out = F_out;
    a.bp = bp_out;
    a.bp_off = bp_off_out;
    a.pt_bin = pt_bin_out;
    a.info = info_out;
    a.L_out = L_out;
    a.stair_bin = stair_bin;
    a.n_stair = n_stair;
    a.status = status_out;
    a.stair_Tlo = stair_Tlo;
    a.stair_E = stair_E;
    hipEvent_t *ev = g_phase_ev[KR_PHASE_MINPLUS];
    return launch_compose(a, w, ev[0] && ev[1] ? ev : nullptr, (hipStream_t)stream) == hipSuccess
               ? KR_OK
               : KR_EHIP;
}

kr_status kr_extract_schedule(int32_t n_parts, int32_t n_bins, const int32_t *bp,
                              const int32_t *bp_off, const int32_t *pt_bin,
                              const int64_t *off, const double *T,
                              const double *E, const int32_t *bins, int32_t n_q,
                              const int32_t *cand_idx, int32_t *choice_out,
                              int32_t *choice_cand_out, double *T_out, double *E_out,
                              int32_t *ok_out, void *stream)
{
    if (n_parts < 1 || n_bins < 2 || n_q < 0 || !bp || !pt_bin || !off || !T || !E ||
        (n_q > 0 && (!bins || !choice_out || !T_out || !E_out || !ok_out)) ||
        (cand_idx && !choice_cand_out))
        return KR_EINVAL;
    ExtractArgs a;
    a.P = n_parts;
    a.B = n_bins;
    a.n_q = n_q;
    a.bp = bp;
    a.bp_off = bp_off;
    a.pt_bin = pt_bin;
    a.bins = bins;
    a.cand_idx = cand_idx;
    a.off = off;
    a.T = T;
    a.E = E;
    a.choice = choice_out;
    a.choice_cand = choice_cand_out;
    a.ok = ok_out;
    a.T_out = T_out;
    a.E_out = E_out;
    return launch_extract(a, (hipStream_t)stream) == hipSuccess ? KR_OK : KR_EHIP;
}

// Workspace of the microbatch frontier; every pointer is null when base is null.
struct MbWs {
    int64_t *seg, *front_off;
    double *slot_T, *slot_E, *front_T, *front_E;
    int32_t *slot_choice, *front_idx;
    MbGridWs g;
    void *pws;
    size_t pws_bytes;
};

static MbWs carve_mb(Carve &c, int K, int F, int B)
{
    MbWs w;
    const int64_t S = (int64_t)F * B;
    w.seg = c.take<int64_t>(2);
    w.front_off = c.take<int64_t>(2);
    w.slot_T = c.take<double>(S);
    w.slot_E = c.take<double>(S);
    w.front_T = c.take<double>(S);
    w.front_E = c.take<double>(S);
    w.slot_choice = c.take<int32_t>((size_t)S * K);
    w.front_idx = c.take<int32_t>(S);
    w.g.ob2 = c.take<int32_t>(S);
    w.g.oarg = c.take<int32_t>(S);
    w.g.oe = c.take<double>(S);
    w.g.F = c.take<double>(2 * S);
    w.g.bp = c.take<int32_t>((size_t)S * K);
    w.g.stair = c.take<int32_t>(S);
    w.pws_bytes = kr_pareto_filter_workspace(S, 1);
    w.pws = c.take<char>(w.pws_bytes);
    return w;
}

size_t kr_microbatch_frontier_workspace(int32_t n_types, int32_t n_freq, int64_t n_points,
                                        int32_t n_seq, int32_t n_bins)
{
    if (n_types < 1 || n_types > KR_MB_MAX_TYPES || n_freq < 1 || n_points < 0 || n_seq < 1 ||
        n_seq > KR_MB_MAX_SEQ || n_bins < 2)
        return 0;
    Carve c(nullptr);
    carve_mb(c, n_types, n_freq, n_bins);
    return c.used;
}

kr_status kr_microbatch_frontier(int32_t n_types, int32_t n_freq, const int64_t *seg_off,
                                 const double *T, const double *E, int64_t n_points,
                                 int32_t n_seq, const int32_t *seq, int32_t n_comp,
                                 const double *comp_T, const double *comp_E, int32_t n_bins,
                                 int64_t cap, double *out_T, double *out_E, int32_t *out_f,
                                 int32_t *out_choice, int64_t *n_out, void *ws, size_t ws_bytes,
                                 void *stream)
{
    const size_t need = kr_microbatch_frontier_workspace(n_types, n_freq, n_points, n_seq, n_bins);
    if (need == 0 || !seg_off || (n_points > 0 && (!T || !E)) || !seq || n_comp < 0 ||
        (n_comp > 0 && (!comp_T || !comp_E)) || cap < 0 ||
        (cap > 0 && (!out_T || !out_E || !out_f || !out_choice)) || !n_out || !ws)
        return KR_EINVAL;
    if (ws_bytes < need) return KR_ECAPACITY;
    MbArgs a;
    a.K = n_types;
    a.F = n_freq;
    a.B = n_bins;
    a.n_seq = n_seq;
    a.n_comp = n_comp;
    a.seg_off = seg_off;
    a.T = T;
    a.E = E;
    a.comp_T = comp_T;
    a.comp_E = comp_E;
    int32_t cnt[KR_MB_MAX_TYPES] = {0}, uidx[KR_MB_MAX_TYPES];
    for (int i = 0; i < n_seq; ++i) {
        if (seq[i] < 0 || seq[i] >= n_types) return KR_EINVAL;
        ++cnt[seq[i]];
    }
    a.Ku = 0;
    for (int t = 0; t < n_types; ++t)
        if (cnt[t] > 0) {
            uidx[t] = a.Ku;
            a.used[a.Ku] = t;
            a.count[a.Ku] = cnt[t];
            ++a.Ku;
        }
    for (int i = 0; i < n_seq; ++i) a.seq_u[i] = (uint8_t)uidx[seq[i]];
    hipStream_t st = (hipStream_t)stream;
    Carve c(ws);
    MbWs w = carve_mb(c, n_types, n_freq, n_bins);
    a.slot_T = w.slot_T;
    a.slot_E = w.slot_E;
    a.slot_choice = w.slot_choice;
    if (launch_mb_grid(a, w.g, st) != hipSuccess) return KR_EHIP;
    const int64_t S = (int64_t)n_freq * n_bins;
    if (launch_mb_seg(w.seg, S, st) != hipSuccess) return KR_EHIP;
    const kr_status rc = kr_pareto_filter(S, w.slot_T, w.slot_E, w.seg, 1, S, w.front_off,
                                          w.front_idx, w.front_T, w.front_E, nullptr, w.pws,
                                          w.pws_bytes, stream);
    if (rc != KR_OK) return rc;
    return launch_mb_gather(a, w.front_off, w.front_idx, cap, out_T, out_E, out_f, out_choice,
                            n_out, st) == hipSuccess
               ? KR_OK
               : KR_EHIP;
}

// Workspace of the enumerating microbatch frontier.
struct MbEnumWs {
    int64_t *base, *seg, *front_off;
    int32_t *status, *front_idx;
    double *slot_T, *slot_E, *front_T, *front_E;
    void *pws;
    size_t pws_bytes;
};

static MbEnumWs carve_mb_enum(Carve &c, int F, int64_t slots)
{
    MbEnumWs w;
    w.base = c.take<int64_t>(F + 1);
    w.seg = c.take<int64_t>(2);
    w.front_off = c.take<int64_t>(2);
    w.status = c.take<int32_t>(1);
    w.front_idx = c.take<int32_t>(slots);
    w.slot_T = c.take<double>(slots);
    w.slot_E = c.take<double>(slots);
    w.front_T = c.take<double>(slots);
    w.front_E = c.take<double>(slots);
    w.pws_bytes = kr_pareto_filter_workspace(slots, 1);
    w.pws = c.take<char>(w.pws_bytes);
    return w;
}

size_t kr_microbatch_enumerate_workspace(int32_t n_types, int32_t n_freq, int64_t n_configs)
{
    if (n_types < 1 || n_types > KR_MB_MAX_TYPES || n_freq < 1 || n_configs < 1 ||
        n_configs > INT32_MAX)
        return 0;
    Carve c(nullptr);
    carve_mb_enum(c, n_freq, n_configs);
    return c.used;
}

kr_status kr_microbatch_enumerate(int32_t n_types, int32_t n_freq, const int64_t *seg_off,
                                  const double *T, const double *E, int32_t n_seq,
                                  const int32_t *seq, int32_t n_comp, const double *comp_T,
                                  const double *comp_E, int64_t n_configs, int64_t cap,
                                  double *out_T, double *out_E, int32_t *out_f,
                                  int32_t *out_choice, int64_t *n_out, int32_t *status_out,
                                  void *ws, size_t ws_bytes, void *stream)
{
    const size_t need = kr_microbatch_enumerate_workspace(n_types, n_freq, n_configs);
    if (need == 0 || !seg_off || !T || !E || !seq || n_seq < 1 || n_seq > KR_MB_MAX_SEQ ||
        n_comp < 0 || (n_comp > 0 && (!comp_T || !comp_E)) || cap < 0 ||
        (cap > 0 && (!out_T || !out_E || !out_f || !out_choice)) || !n_out || !status_out || !ws)
        return KR_EINVAL;
    if (ws_bytes < need) return KR_ECAPACITY;
    MbArgs a;
    a.K = n_types;
    a.F = n_freq;
    a.B = 0;
    a.n_seq = n_seq;
    a.n_comp = n_comp;
    a.seg_off = seg_off;
    a.T = T;
    a.E = E;
    a.comp_T = comp_T;
    a.comp_E = comp_E;
    int32_t cnt[KR_MB_MAX_TYPES] = {0}, uidx[KR_MB_MAX_TYPES];
    for (int i = 0; i < n_seq; ++i) {
        if (seq[i] < 0 || seq[i] >= n_types) return KR_EINVAL;
        ++cnt[seq[i]];
    }
    a.Ku = 0;
    for (int t = 0; t < n_types; ++t)
        if (cnt[t] > 0) {
            uidx[t] = a.Ku;
            a.used[a.Ku] = t;
            a.count[a.Ku] = cnt[t];
            ++a.Ku;
        }
    for (int i = 0; i < n_seq; ++i) a.seq_u[i] = (uint8_t)uidx[seq[i]];
    hipStream_t st = (hipStream_t)stream;
    Carve c(ws);
    MbEnumWs w = carve_mb_enum(c, n_freq, n_configs);
    a.slot_T = w.slot_T;
    a.slot_E = w.slot_E;
    a.slot_choice = nullptr;
    if (launch_mb_enum(a, w.base, n_configs, w.status, st) != hipSuccess) return KR_EHIP;
    if (launch_mb_seg(w.seg, n_configs, st) != hipSuccess) return KR_EHIP;
    const kr_status rc = kr_pareto_filter(n_configs, w.slot_T, w.slot_E, w.seg, 1, n_configs,
                                          w.front_off, w.front_idx, w.front_T, w.front_E, nullptr,
                                          w.pws, w.pws_bytes, stream);
    if (rc != KR_OK) return rc;
    if (launch_mb_enum_gather(a, w.base, w.status, w.front_off, w.front_idx, cap, out_T, out_E,
                              out_f, out_choice, n_out, n_configs, st) != hipSuccess)
        return KR_EHIP;
    return hipMemcpyAsync(status_out, w.status, sizeof(int32_t), hipMemcpyDeviceToDevice, st) ==
                   hipSuccess
               ? KR_OK
               : KR_EHIP;
}

kr_status kr_decode_candidates(const kr_space *space, const int32_t *idx, int64_t n,
                               int32_t *f_out, int32_t *pos_out, int32_t *sm_out, void *stream)
{
    if (!space_ok(space) || n < 0 || (n > 0 && (!idx || !f_out || !pos_out || !sm_out)))
        return KR_EINVAL;
    DecodeArgs d;
    d.idx = idx;
    d.n = n;
    d.f_out = f_out;
    d.pos_out = pos_out;
    d.sm_out = sm_out;
    d.M = space->n_comm;
    d.S = space->n_sm;
    d.n_pos = space->n_pos;
    d.F = space->n_freq;
    const int64_t cf = cand_per_freq(space);
    if (cf * space->n_freq > 0x7FFFFFFF) return KR_EUNSUPPORTED;
    d.Cf = (int)cf;
    return launch_decode(d, (hipStream_t)stream) == hipSuccess ? KR_OK : KR_EHIP;
}

size_t kr_hvi_scores_workspace(int32_t n_seg, int64_t n_obs)
{
    if (n_seg < 1 || n_obs < 1) return 0;
    Carve c(nullptr);
    c.take<double>(3 * n_obs);
    c.take<double>(3 * n_obs);
    c.take<int32_t>(3 * (int64_t)n_seg);
    return c.used;
}

kr_status kr_hvi_scores(int32_t n_seg, int64_t n_cand, const int64_t *cand_off,
                        const double *T_hat, const double *E_hat, int64_t n_obs,
                        const int64_t *obs_off, const double *T_obs, const double *E_obs,
                        double p_static, double *hvi_out, double *hv_out, double *ref_out,
                        int32_t *status_out, void *ws, size_t ws_bytes, void *stream)
{
    const size_t need = kr_hvi_scores_workspace(n_seg, n_obs);
    if (need == 0 || n_cand < 0 || !cand_off || !obs_off || !T_obs || !E_obs || !hv_out ||
        !ref_out || !status_out || !ws || !(p_static == p_static) ||
        (n_cand > 0 && (!T_hat || !E_hat || !hvi_out)))
        return KR_EINVAL;
    if (ws_bytes < need) return KR_ECAPACITY;
    Carve c(ws);
    HviArgs a;
    a.n_seg = n_seg;
    a.n_cand = n_cand;
    a.n_obs = n_obs;
    a.cand_off = cand_off;
    a.obs_off = obs_off;
    a.T_hat = T_hat;
    a.E_hat = E_hat;
    a.T_obs = T_obs;
    a.E_obs = E_obs;
    a.p_static = p_static;
    a.fr_T = c.take<double>(3 * n_obs);
    a.fr_E = c.take<double>(3 * n_obs);
    a.fr_n = c.take<int32_t>(3 * (int64_t)n_seg);
    a.hvi = hvi_out;
    a.hv = hv_out;
    a.ref = ref_out;
    a.status = status_out;
    return launch_hvi(a, g_phase_ev[KR_PHASE_HVI], (hipStream_t)stream) == hipSuccess ? KR_OK
                                                                                  : KR_EHIP;
}

kr_status kr_uncertainty(int32_t n_members, int64_t n, const double *T_m, const double *E_m,
                         double *unc_out, void *stream)
{
    if (n_members < 1 || n_members > 64 || n < 0 || (n > 0 && (!T_m || !E_m || !unc_out)))
        return KR_EINVAL;
    return launch_uncertainty(n_members, n, T_m, E_m, unc_out, g_phase_ev[KR_PHASE_UNC],
                              (hipStream_t)stream) ==
                   hipSuccess
               ? KR_OK
               : KR_EHIP;
}

size_t kr_select_batch_workspace(int32_t n_seg, int64_t n_cand)
{
    if (n_seg < 1 || n_cand < 0) return 0;
    const int64_t tiles = n_cand / KR_SEL_TILE + n_seg;
    Carve c(nullptr);
    c.take<int64_t>(n_seg + 1);
    c.take<int32_t>(1);
    c.take<uint64_t>(tiles * 4 * KR_SEL_LIST);
    c.take<int32_t>(tiles * 4 * KR_SEL_LIST);
    return c.used;
}

kr_status kr_select_batch(int32_t n_seg, int64_t n_cand, const int64_t *cand_off,
                          const double *score, const double *unc, const int64_t *obs_off,
                          const int64_t *obs_idx, int32_t k1, int32_t k2, int32_t k3, int32_t k,
                          int64_t *sel_out, int32_t *count_out, int32_t *status_out, void *ws,
                          size_t ws_bytes, void *stream)
{
    const size_t need = kr_select_batch_workspace(n_seg, n_cand);
    if (need == 0 || !cand_off || !obs_off || !obs_idx || !count_out || !status_out || !ws ||
        (n_cand > 0 && !score) || k1 < 0 || k2 < 0 || k3 < 0 ||
        (int64_t)k1 + k2 + k3 > k || k > KR_SELECT_MAX_K || (k > 0 && !sel_out))
        return KR_EINVAL;
    if (ws_bytes < need) return KR_ECAPACITY;
    Carve c(ws);
    SelArgs a;
    a.n_seg = n_seg;
    a.n_cand = n_cand;
    a.cand_off = cand_off;
    a.obs_off = obs_off;
    a.obs_idx = obs_idx;
    a.score = score;
    a.unc = unc;
    a.k[0] = k1;
    a.k[1] = k2;
    a.k[2] = k3;
    a.k[3] = k;
    a.npass = unc ? 4 : 3;
    a.max_tiles = n_cand / KR_SEL_TILE + n_seg;
    a.tile_off = c.take<int64_t>(n_seg + 1);
    a.flag = c.take<int32_t>(1);
    a.part_key = c.take<uint64_t>(a.max_tiles * 4 * KR_SEL_LIST);
    a.part_idx = c.take<int32_t>(a.max_tiles * 4 * KR_SEL_LIST);
    a.sel = sel_out;
    a.count = count_out;
    a.status = status_out;
    return launch_select(a, g_phase_ev[KR_PHASE_SELECT], (hipStream_t)stream) == hipSuccess
               ? KR_OK
               : KR_EHIP;
}

size_t kr_compare_frontiers_workspace(void)
{
    Carve c(nullptr);
    c.take<double>(3 * KR_CMP_BLOCKS);
    c.take<double>(5 * KR_CMP_BLOCKS);
    return c.used;
}

kr_status kr_compare_frontiers(int64_t nA, const double *TA, const double *EA, int64_t nB,
                               const double *TB, const double *EB, double *out, void *ws,
                               size_t ws_bytes, void *stream)
{
    if (nA < 1 || nB < 1 || !TA || !EA || !TB || !EB || !out || !ws) return KR_EINVAL;
    if (ws_bytes < kr_compare_frontiers_workspace()) return KR_ECAPACITY;
    Carve c(ws);
    CmpArgs a;
    a.nA = nA;
    a.nB = nB;
    a.TA = TA;
    a.EA = EA;
    a.TB = TB;
    a.EB = EB;
    const int64_t need = (std::max(nA, nB) + KR_BLOCK * 4 - 1) / (KR_BLOCK * 4);
    a.blocks = (int)std::min<int64_t>(KR_CMP_BLOCKS, std::max<int64_t>(1, need));
    a.part = c.take<double>(3 * KR_CMP_BLOCKS);
    a.part2 = c.take<double>(5 * KR_CMP_BLOCKS);
    a.out = out;
    return launch_compare(a, (hipStream_t)stream) == hipSuccess ? KR_OK : KR_EHIP;
}

size_t kr_launch_timing_frontier_workspace(int64_t n_inst)
{
    if (n_inst < 0 || n_inst > INT32_MAX) return 0;
    Carve c(nullptr);
    c.take<int32_t>(2);
    c.take<int32_t>(2 * std::max<int64_t>(n_inst, 1));
    return c.used;
}

kr_status kr_launch_timing_frontier(int64_t n_inst, int32_t I, int32_t J, const int32_t *kind,
                                    const double *ops, double p_static, int32_t kmax,
                                    int32_t out_cap, double *out_T, double *out_E,
                                    int32_t *out_sched, int32_t *out_n, int32_t *status_out,
                                    void *ws, size_t ws_bytes, void *stream)
{
    if (n_inst < 0 || n_inst > INT32_MAX || I < 0 || J < 0 || I > KR_DP_MAX_OPS ||
        J > KR_DP_MAX_OPS || I + J < 1 || !kind || kmax < 0 || kmax > KR_DP_MAX_K ||
        out_cap < 1 || out_cap > 64 || !status_out || !(p_static == p_static) ||
        (n_inst > 0 && (!ops || !out_T || !out_E || !out_n)) || !ws)
        return KR_EINVAL;
    if (ws_bytes < kr_launch_timing_frontier_workspace(n_inst)) return KR_ECAPACITY;
    DpArgs a;
    std::memset(&a, 0, sizeof(a));
    a.n_inst = n_inst;
    a.I = I;
    a.J = J;
    a.kmax = kmax;
    a.out_cap = out_cap;
    for (int o = 0; o < I + J; ++o) {
        if (kind[o] != 0 && kind[o] != 1) return KR_EINVAL;
        a.kind[o] = (int8_t)kind[o];
    }
    for (int i = I - 1; i >= 0; --i) a.run1[i] = kind[i] == 0 ? (int8_t)(a.run1[i + 1] + 1) : 0;
    for (int j = J - 1; j >= 0; --j)
        a.run2[j] = kind[I + j] == 0 ? (int8_t)(a.run2[j + 1] + 1) : 0;
    a.ops = ops;
    a.p_static = p_static;
    a.out_T = out_T;
    a.out_E = out_E;
    a.out_sched = out_sched;
    a.out_n = out_n;
    a.status = status_out;
    // first pass: a budget that lets many instances share a compute unit's LDS
    a.arena_s = 384;
    a.cand_s = 128;
    Carve c(ws);
    a.retry_n = c.take<int32_t>(2);
    a.retry = c.take<int32_t>(2 * std::max<int64_t>(n_inst, 1));
    return launch_dp(a, (hipStream_t)stream) == hipSuccess ? KR_OK : KR_EHIP;
}

int32_t kr_hv_converged(int32_t n, const double *hv_history, int32_t R, double eps)
{
    if (R < 1 || !hv_history || n - 1 < R) return 0;
    double s = 0.0;
    for (int b = n - R; b < n; ++b) {
        if (!(hv_history[b - 1] != 0.0)) return 0;
        s = s + (hv_history[b] - hv_history[b - 1]) / hv_history[b - 1];
    }
    return s / R < eps ? 1 : 0;
}

kr_status kr_set_phase_events(int32_t phase, void *start_event, void *stop_event)
{
    if (phase < 0 || phase > 5) return KR_EINVAL;
    g_phase_ev[phase][0] = (hipEvent_t)start_event;
    g_phase_ev[phase][1] = (hipEvent_t)stop_event;
    return KR_OK;
}

const char *kr_status_string(kr_status status)
{
    switch (status) {
    case KR_OK: return "ok";
    case KR_EINVAL: return "invalid argument";
    case KR_ENONFINITE: return "non-finite or negative input";
    case KR_ECAPACITY: return "workspace or output capacity too small";
    case KR_EHIP: return "HIP runtime error";
    case KR_EUNSUPPORTED: return "shape exceeds the kernels' on-chip limits";
    default: return "unknown status";
    }
}

}  // extern "C"
