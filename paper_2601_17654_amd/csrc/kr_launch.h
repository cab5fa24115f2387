// Launch arguments and host-side launchers of the library's kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kr {

struct EvalArgs {
    const double *t, *pw, *tc, *pc;
    double *T_out, *E_out;  // unfused evaluation only
    int P, N, M, F, S, n_pos, n_pp;
    int Cf;                 // candidates per frequency
    int64_t C;              // candidates per partition
    double p_static;
    int slab_doubles;       // LDS doubles of the table slab
    int pair_doubles;       // LDS doubles holding the position-pair table
    int tile;               // fused: candidates per tile
    int tiles_per_freq;     // fused: tiles per frequency
    int cpt;                // fused: candidates per thread (tile <= 256 * cpt)
};

// Tile-local frontiers written by the fused kernel or the pareto tile kernel.
struct TileOut {
    double *T, *E;
    int32_t *I;
    int32_t *cnt;           // [segments * tiles_per_seg]
    int64_t tiles_per_seg;  // fused path: F * tiles_per_freq
    int nb;                 // time buckets of the prefilter
};

struct DecodeArgs {
    const int32_t *idx;
    int64_t n;
    int32_t *f_out, *pos_out, *sm_out;
    int M, S, n_pos, F, Cf;
};

// Segmented frontier: layout of tiles inside segments.
struct SegLayout {
    const int64_t *seg_off;   // [n_seg + 1] element offsets
    const int64_t *tile_base; // [n_seg + 1] first tile of each segment
    int n_seg;
    int tile;                 // elements per tile
    int tiles_per_group;      // tiles per frequency group (fused), else 1
    int64_t group_elems;      // elements per group (fused: candidates per frequency)
};

struct PointBufs {
    double *T, *E;
    int32_t *I;
};

hipError_t launch_eval(const EvalArgs &a, hipStream_t st);
hipError_t launch_eval_filter(const EvalArgs &a, const TileOut &o, hipStream_t st);
hipError_t launch_decode(const DecodeArgs &d, hipStream_t st);

// pareto.hip
hipError_t launch_uniform_layout(int64_t *seg_off, int64_t *tile_base, int n_seg,
                                 int64_t seg_len, int64_t tiles_per_seg, hipStream_t st);
hipError_t launch_tile_layout(const int64_t *seg_off, int64_t *tile_base, int n_seg, int tile,
                              hipStream_t st);
hipError_t launch_pareto_tiles(const double *T, const double *E, const SegLayout &L,
                               int64_t n_tiles_bound, const TileOut &o, int cpt, hipStream_t st);
hipError_t launch_merge_level(const SegLayout &L, int level, int64_t max_tiles,
                              const PointBufs &in, const int32_t *cnt_in, const PointBufs &out,
                              int32_t *cnt_out, uint8_t *flags, hipStream_t st);
hipError_t launch_finish(const SegLayout &L, const PointBufs &fin, const int32_t *cnt,
                         int64_t cap, int64_t *out_off, int32_t *out_idx, double *out_T,
                         double *out_E, hipStream_t st);

// compose.hip
struct ComposeWs {
    double *tmin, *range;  // [P]
    int64_t *Mk, *Lk, *eoff;  // [P], [P], [P+1]
    uint64_t *ebits;       // [B + P]
    int32_t *earg;         // [B + P]
    int32_t *ob2, *oarg;   // [B + P] occupied offsets / point index
    double *oe;            // [B + P]
    int32_t *occ;          // [P]
    double *F0, *F1;       // [B]
};
struct ComposeArgs {
    int P, B;
    double delta_in;
    const int64_t *off;
    const double *T, *E;
    double *F_out;
    int32_t *bp, *pt_bin;
    double *info;
    int32_t *L_out, *stair_bin, *n_stair, *status;
    double *stair_Tlo, *stair_E;
};
hipError_t launch_compose(const ComposeArgs &a, const ComposeWs &w, hipStream_t st);

struct ExtractArgs {
    int P, B, n_q;
    const int32_t *bp, *pt_bin, *bins, *cand_idx;
    const int64_t *off;
    const double *T, *E;
    int32_t *choice, *choice_cand, *ok;
    double *T_out, *E_out;
};
hipError_t launch_extract(const ExtractArgs &a, hipStream_t st);

}  // namespace kr
