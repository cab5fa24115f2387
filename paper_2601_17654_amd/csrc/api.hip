// C ABI of libkareus_mi355x.so: argument checks, workspace layout and launch order.
// Declarations and contracts: include/kareus.h.
#include <algorithm>
#include <cstring>

#include "../../include/kareus.h"
#include "kr_launch.h"

using namespace kr;

namespace {

constexpr int kTile = 2048;        // points per tile of the stand-alone filter
constexpr int kBuckets = 512;      // time buckets of the tile prefilter
constexpr size_t kLdsBudget = 65536;
constexpr size_t kAlign = 256;

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
    a->slab_doubles = (int)(2 * a->N * S1 + 2 * S1 * (a->N + 1) + 2 * a->M * a->S);
    a->pair_doubles = a->M == 2 ? (a->n_pp * 4 + 7) / 8 : 0;
    size_t lds = (size_t)(a->slab_doubles + a->pair_doubles) * 8;
    if (lds > kLdsBudget) return false;
    if (!fused) return true;
    static const int cpts[] = {1, 2, 4, 5, 8};
    int pick = 4;
    for (int i = 0; i < 5; ++i)
        if ((int64_t)256 * cpts[i] >= a->Cf) {
            pick = i;
            break;
        }
    for (; pick >= 0; --pick) {
        const int tile = (int)std::min<int64_t>(a->Cf, 256 * cpts[pick]);
        if (lds + (size_t)kBuckets * 8 + (size_t)tile * 20 <= kLdsBudget) {
            a->cpt = cpts[pick];
            a->tile = tile;
            a->tiles_per_freq = (a->Cf + tile - 1) / tile;
            return true;
        }
    }
    return false;
}

int levels_for(int64_t tiles)
{
    int l = 0;
    while (((int64_t)1 << l) < tiles) ++l;
    return l;
}

struct FilterWs {
    int64_t *seg_off, *tile_base;
    int32_t *cnt[2];
    PointBufs buf[2];
    uint8_t *flags;
};

FilterWs carve_filter(Carve &c, int64_t n_total, int n_seg, int64_t n_tiles, bool own_seg_off)
{
    FilterWs w;
    w.seg_off = own_seg_off ? c.take<int64_t>(n_seg + 1) : nullptr;
    w.tile_base = c.take<int64_t>(n_seg + 1);
    for (int i = 0; i < 2; ++i) w.cnt[i] = c.take<int32_t>(std::max<int64_t>(n_tiles, 1));
    for (int i = 0; i < 2; ++i) {
        w.buf[i].T = c.take<double>(std::max<int64_t>(n_total, 1));
        w.buf[i].E = c.take<double>(std::max<int64_t>(n_total, 1));
        w.buf[i].I = c.take<int32_t>(std::max<int64_t>(n_total, 1));
    }
    w.flags = c.take<uint8_t>(std::max<int64_t>(n_total, 1));
    return w;
}

// Merge the tile frontiers of every segment level by level, then write the output.
kr_status merge_and_finish(const SegLayout &L, FilterWs &w, int64_t max_tiles, int64_t cap,
                           int64_t *out_off, int32_t *out_idx, double *out_T, double *out_E,
                           hipStream_t st)
{
    const int levels = levels_for(max_tiles);
    for (int l = 0; l < levels; ++l) {
        if (launch_merge_level(L, l, max_tiles, w.buf[l % 2], w.cnt[l % 2], w.buf[(l + 1) % 2],
                               w.cnt[(l + 1) % 2], w.flags, st) != hipSuccess)
            return KR_EHIP;
    }
    if (launch_finish(L, w.buf[levels % 2], w.cnt[levels % 2], cap, out_off, out_idx, out_T,
                      out_E, st) != hipSuccess)
        return KR_EHIP;
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
                                void *stream)
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
    return launch_eval(a, (hipStream_t)stream) == hipSuccess ? KR_OK : KR_EHIP;
}

size_t kr_pareto_filter_workspace(int64_t n_total, int32_t n_seg, int64_t max_seg_len)
{
    if (n_total < 0 || n_seg < 0 || max_seg_len < 0) return 0;
    const int64_t n_tiles = (n_total + kTile - 1) / kTile + n_seg;
    Carve c(nullptr);
    carve_filter(c, n_total, n_seg, n_tiles, false);
    return c.used;
}

kr_status kr_pareto_filter(int64_t n_total, const double *T, const double *E,
                           const int64_t *seg_off, int32_t n_seg, int64_t max_seg_len, int64_t cap,
                           int64_t *out_off, int32_t *out_idx, double *out_T, double *out_E,
                           void *ws, size_t ws_bytes, void *stream)
{
    if (n_total < 0 || n_seg < 0 || max_seg_len < 0 || max_seg_len > 0x7FFFFFFF || cap < 0 ||
        !seg_off || !out_off || (n_total > 0 && (!T || !E)) ||
        (cap > 0 && (!out_idx || !out_T || !out_E)) || !ws)
        return KR_EINVAL;
    if (ws_bytes < kr_pareto_filter_workspace(n_total, n_seg, max_seg_len)) return KR_ECAPACITY;
    hipStream_t st = (hipStream_t)stream;
    const int64_t n_tiles = (n_total + kTile - 1) / kTile + n_seg;
    Carve c(ws);
    FilterWs w = carve_filter(c, n_total, n_seg, n_tiles, false);
    SegLayout L;
    L.seg_off = seg_off;
    L.tile_base = w.tile_base;
    L.n_seg = n_seg;
    L.tile = kTile;
    L.tiles_per_group = 1;
    L.group_elems = kTile;
    if (n_seg > 0 && launch_tile_layout(seg_off, w.tile_base, n_seg, kTile, st) != hipSuccess)
        return KR_EHIP;
    TileOut o;
    o.T = w.buf[0].T;
    o.E = w.buf[0].E;
    o.I = w.buf[0].I;
    o.cnt = w.cnt[0];
    o.tiles_per_seg = 0;
    o.nb = kBuckets;
    if (n_seg > 0 && launch_pareto_tiles(T, E, L, n_tiles, o, kTile / 256, st) != hipSuccess)
        return KR_EHIP;
    const int64_t max_tiles = (max_seg_len + kTile - 1) / kTile;
    return merge_and_finish(L, w, max_tiles, cap, out_off, out_idx, out_T, out_E, st);
}

size_t kr_evaluate_and_filter_workspace(const kr_space *space)
{
    EvalArgs a;
    if (!space_ok(space) || !eval_plan(space, true, &a)) return 0;
    const int64_t tiles = (int64_t)a.P * a.F * a.tiles_per_freq;
    Carve c(nullptr);
    carve_filter(c, (int64_t)a.P * a.C, a.P, tiles, true);
    return c.used;
}

kr_status kr_evaluate_and_filter(const kr_space *space, const double *t, const double *pw,
                                 const double *tc, const double *pc, int64_t cap, int64_t *out_off,
                                 int32_t *out_idx, double *out_T, double *out_E, void *ws,
                                 size_t ws_bytes, void *stream)
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
    const int64_t tiles_per_seg = (int64_t)a.F * a.tiles_per_freq;
    Carve c(ws);
    FilterWs w = carve_filter(c, (int64_t)a.P * a.C, a.P, tiles_per_seg * a.P, true);
    if (launch_uniform_layout(w.seg_off, w.tile_base, a.P, a.C, tiles_per_seg, st) != hipSuccess)
        return KR_EHIP;
    TileOut o;
    o.T = w.buf[0].T;
    o.E = w.buf[0].E;
    o.I = w.buf[0].I;
    o.cnt = w.cnt[0];
    o.tiles_per_seg = tiles_per_seg;
    o.nb = kBuckets;
    if (launch_eval_filter(a, o, st) != hipSuccess) return KR_EHIP;
    SegLayout L;
    L.seg_off = w.seg_off;
    L.tile_base = w.tile_base;
    L.n_seg = a.P;
    L.tile = a.tile;
    L.tiles_per_group = a.tiles_per_freq;
    L.group_elems = a.Cf;
    return merge_and_finish(L, w, tiles_per_seg, cap, out_off, out_idx, out_T, out_E, st);
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
    c.take<uint64_t>(B + P);
    c.take<int32_t>(B + P);
    c.take<int32_t>(B + P);
    c.take<int32_t>(B + P);
    c.take<double>(B + P);
    c.take<int32_t>(P);
    c.take<double>(B);
    c.take<double>(B);
    return c.used;
}

kr_status kr_compose_frontiers(int32_t n_parts, const int64_t *off, const double *T,
                               const double *E, int32_t n_bins, double delta, double *F_out,
                               int32_t *bp_out, int32_t *pt_bin_out, double *info_out,
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
    w.ebits = c.take<uint64_t>(B + P);
    w.earg = c.take<int32_t>(B + P);
    w.ob2 = c.take<int32_t>(B + P);
    w.oarg = c.take<int32_t>(B + P);
    w.oe = c.take<double>(B + P);
    w.occ = c.take<int32_t>(P);
    w.F0 = c.take<double>(B);
    w.F1 = c.take<double>(B);
    ComposeArgs a;
    a.P = n_parts;
    a.B = n_bins;
    a.delta_in = delta;
    a.off = off;
    a.T = T;
    a.E = E;
    a.F_out = F_out;
    a.bp = bp_out;
    a.pt_bin = pt_bin_out;
    a.info = info_out;
    a.L_out = L_out;
    a.stair_bin = stair_bin;
    a.n_stair = n_stair;
    a.status = status_out;
    a.stair_Tlo = stair_Tlo;
    a.stair_E = stair_E;
    return launch_compose(a, w, (hipStream_t)stream) == hipSuccess ? KR_OK : KR_EHIP;
}

kr_status kr_extract_schedule(int32_t n_parts, int32_t n_bins, const int32_t *bp,
                              const int32_t *pt_bin, const int64_t *off, const double *T,
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

const char *kr_status_string(kr_status status)
{
    switch (status) {
    case KR_OK: return "ok";
    case KR_EINVAL: return "invalid argument";
    case KR_ECAPACITY: return "workspace or output capacity too small";
    case KR_EHIP: return "HIP runtime error";
    case KR_EUNSUPPORTED: return "shape exceeds the kernels' on-chip limits";
    default: return "unknown status";
    }
}

}  // extern "C"
