// Launch arguments and host-side launchers of the library's kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/kareus.h"

#define KR_FIN_CAP 2560    // points the finalize kernel sorts in LDS
#define KR_PAIR_WAVES 4    // waves per block of the two-comm evaluation kernel
#define KR_FIN_UNITS 2048  // units per segment the finalize kernel's LDS path takes
#define KR_TILE 2048       // points per tile of the stand-alone filter
#define KR_PAD 3           // rows the wave kernel's end-cursor search reads per step
// Power-slab offset (doubles) of the one-wave layout with 32 kernels and 32 SM choices:
// t slab and pad rows, rounded up to keep the second table 16-byte aligned.
#define KR_FIX32_PW (((32 + KR_PAD) * 33 + 1) / 2 * 2)

namespace kr {

struct EvalArgs {
    const double *t, *pw, *tc, *pc;
    double *T_out, *E_out;  // unfused evaluation only
    int P, N, M, F, S, n_pos, n_pp;
    int Cf;                 // candidates per frequency
    int64_t C;              // candidates per partition
    double p_static;
    int lds_doubles;        // dynamic LDS of the launch, in doubles
    // fused evaluation + filter
    int surv_off;           // LDS offset (doubles) of the survivor list
    int nfb, fb;            // frequency blocks per partition, frequencies per block
    int one_comm;           // one comm kernel: thread = (SM choice, run of positions)
    int nchunk, cpt;        // position runs per tile / positions (or candidates) per thread
    int ntiles, tile;       // tiles per frequency; candidates per tile (generic mapping)
    int pf;                 // doubles per thread and table of the register prefetch
    // one wave per slab (one comm kernel, at most 64 SM choices)
    int wave;               // use the wave kernel
    int H, span;            // position runs per SM choice, positions per run
    int R, nch;             // positions per chunk (registers), chunks per run
    int w_pw, w_a0;         // LDS offsets (doubles) of the power slab and the column sums
    int dma16;              // 16-byte direct copies (slab length even, tables 16-byte aligned)
    int wcap;               // candidates the wave filter's LDS scratch holds
    // 32 kernels, 33 launch positions and 32 SM choices (the evaluation stress shape):
    // two runs of 16 and 17 positions per SM choice, one chunk each.  The kernel instance
    // for it takes the sizes, the LDS layout and the validity of all but the last round
    // as compile-time facts
    int fixed32;
    // one wave per slab (two comm kernels, at most 8 SM choices): LDS offsets (doubles)
    // of the power slab, the running sums, the fresh and continuing second-phase
    // records and the filter scratch
    int pair;
    int q_pw, q_ab, q_f, q_c, q_sc;
    int pair_scap;          // most chunk outputs of a slab a wave reduces to its frontier on chip
    // unit slots of the fused launch: points per partition segment, units per segment,
    // points per unit
    int64_t useg, uper, ustride;
};

// Per-unit frontiers written by the fused kernel or the tile kernel.
struct UnitOut {
    double *T, *E;
    int32_t *I;
    int32_t *cnt;  // [units]
};

struct DecodeArgs {
    const int32_t *idx;
    int64_t n;
    int32_t *f_out, *pos_out, *sm_out;
    int M, S, n_pos, F, Cf;
};

// Units of segment g are unit_base[g] .. unit_base[g+1]-1; unit k of segment g has its
// slot at element seg_off[g] + k * unit_stride.
struct SegLayout {
    const int64_t *seg_off;    // [n_seg + 1]
    const int64_t *unit_base;  // [n_seg + 1]
    int n_seg;
    int64_t unit_stride;
};

struct PointBufs {
    double *T, *E;
    int32_t *I;
};

hipError_t launch_eval(const EvalArgs &a, hipStream_t st);
hipError_t launch_eval_filter(const EvalArgs &a, const UnitOut &o, hipStream_t st);
hipError_t launch_eval_filter_wave(const EvalArgs &a, const UnitOut &o, hipStream_t st);
hipError_t launch_eval_filter_pair(const EvalArgs &a, const UnitOut &o, hipStream_t st);
// The wave of a two-comm evaluation block of NW waves that takes launch position p1.
int pair_owner_host(int p1, int NW);
hipError_t launch_decode(const DecodeArgs &d, hipStream_t st);

// pareto.hip
// Both layouts also clear lists[0], which launch_finalize expects to be zero.
hipError_t launch_uniform_layout(int64_t *seg_off, int64_t *unit_base, int n_seg,
                                 int64_t seg_len, int64_t units_per_seg, int32_t *lists,
                                 hipStream_t st);
hipError_t launch_tile_layout(const int64_t *seg_off, int64_t *unit_base, int n_seg, int tile,
                              int32_t *lists, hipStream_t st);
hipError_t launch_pareto_tiles(const double *T, const double *E, const SegLayout &L,
                               int64_t n_units_bound, const UnitOut &o, hipStream_t st);
// lists: 2 * n_seg + 2 ints of scratch, lists[0] zero on entry (cleared by the layout
// launches above)
hipError_t launch_finalize(const SegLayout &L, const PointBufs &buf, const int32_t *ucnt,
                           const PointBufs &fin, int32_t *fcnt, int32_t *runcnt, uint8_t *flags,
                           int32_t *lists, hipStream_t st);
hipError_t launch_output(const SegLayout &L, const PointBufs &fin, const int32_t *fcnt,
                         int64_t cap, int64_t *out_off, int32_t *out_idx, double *out_T,
                         double *out_E, hipStream_t st);

// compose.hip
struct ComposeWs {
    double *tmin, *range;  // [P]
    int64_t *Mk, *Lk, *eoff;  // [P], [P], [P+1]
    int64_t *mmax;            // [1] largest M
    // Per partition k from eoff[k]: the least-energy table over offsets 0 .. M_k + 7
    // (empty past M_k) and the compact list of its occupied offsets.
    uint64_t *ebits;       // [B + 8P]
    int32_t *earg;         // [B + 8P]
    int32_t *ob2, *oarg;   // [B + 8P] occupied offsets / point index
    double *oe;            // [B + 8P]
    int32_t *occ;          // [P]
    double *Fh;            // [P][B] step history of the wavefront min-plus
    int32_t *ticket;       // [1] tile tickets of the wavefront min-plus (reset per call)
    double *chmin;         // [ceil(B / KR_ST_CHUNK)] least value of each staircase chunk
    int32_t *chcnt;        // [ceil(B / KR_ST_CHUNK)] staircase bins of each chunk
};
#define KR_ST_CHUNK 1024   // bins per block of the staircase passes
struct ComposeArgs {
    int P, B;
    double delta_in;
    const int64_t *off;
    const double *T, *E;
    double *F_out;
    int32_t *bp, *pt_bin;
    int32_t *bp_off;  // NULL, or [P][B]: offset of the chosen point (like bp)
    double *info;
    int32_t *L_out, *stair_bin, *n_stair, *status;
    double *stair_Tlo, *stair_E;
};
// check.hip: status = KR_ENONFINITE if some value of the arrays is NaN, infinite or
// negative (-0.0 counts as 0), else KR_OK.
hipError_t launch_check(const double *const *xs, const int64_t *n, int count, int32_t *status,
                        hipStream_t st);

hipError_t launch_compose(const ComposeArgs &a, const ComposeWs &w, hipEvent_t *minplus_ev,
                          hipStream_t st);

struct ExtractArgs {
    int P, B, n_q;
    const int32_t *bp, *pt_bin, *bins, *cand_idx;
    const int32_t *bp_off;  // NULL, or the offsets kr_compose_frontiers recorded
    const int64_t *off;
    const double *T, *E;
    int32_t *choice, *choice_cand, *ok;
    double *T_out, *E_out;
};
hipError_t launch_extract(const ExtractArgs &a, hipStream_t st);

// microbatch.hip
#define KR_MB_MAX_TYPES 32
#define KR_MB_MAX_SEQ 2048
struct MbArgs {
    int K, F, B, Ku, n_seq, n_comp;
    const int64_t *seg_off;
    const double *T, *E;
    const double *comp_T, *comp_E;
    int32_t used[KR_MB_MAX_TYPES];   // used types, in type order
    int32_t count[KR_MB_MAX_TYPES];  // their repeat counts
    uint8_t seq_u[KR_MB_MAX_SEQ];    // used-type index of each partition
    double *slot_T, *slot_E;         // [F * B]
    int32_t *slot_choice;            // [F * B][K]
};
// Per-frequency workspace of the grid microbatch frontier (region f of each array is
// frequency f's): the occupied offsets of the type being binned [B] (offset, least
// energy, point), the composite arrays of two steps [2][B], the back-pointers [K][B] and
// the staircase bins [B].
struct MbGridWs {
    int32_t *ob2, *oarg;
    double *oe, *F;
    int32_t *bp, *stair;
};
hipError_t launch_mb_grid(const MbArgs &a, const MbGridWs &w, hipStream_t st);
hipError_t launch_mb_seg(int64_t *seg, int64_t n, hipStream_t st);
hipError_t launch_mb_gather(const MbArgs &a, const int64_t *front_off, const int32_t *front_idx,
                            int64_t cap, double *out_T, double *out_E, int32_t *out_f,
                            int32_t *out_choice, int64_t *n_out, hipStream_t st);
// Enumeration: base [F + 1] configuration totals, status [1]; slot_T / slot_E [slots].
hipError_t launch_mb_enum(const MbArgs &a, int64_t *base, int64_t slots, int32_t *status,
                          hipStream_t st);
hipError_t launch_mb_enum_gather(const MbArgs &a, const int64_t *base, const int32_t *status,
                                 const int64_t *front_off, const int32_t *front_idx, int64_t cap,
                                 double *out_T, double *out_E, int32_t *out_f, int32_t *out_choice,
                                 int64_t *n_out, int64_t slots, hipStream_t st);

// mbo.hip: scores and batch selection of the Bayesian optimisation (Section 4.3,
// Algorithm 1).
#define KR_HVI_TILE 1024  // candidates per block of the score kernel
#define KR_SEL_TILE 32768  // candidates per block of the selection tile kernel
#define KR_SEL_LIST 64    // entries of a wave's top list (one per lane)

struct HviArgs {
    int32_t n_seg;
    int64_t n_cand, n_obs;
    const int64_t *cand_off, *obs_off;
    const double *T_hat, *E_hat, *T_obs, *E_obs;
    double p_static;
    double *fr_T, *fr_E;  // [3][n_obs]: variant v's frontier of partition g at obs_off[g]
    int32_t *fr_n;        // [n_seg][3] frontier sizes, -1 for a partition with bad counts
    double *hvi, *hv, *ref;
    int32_t *status;
};
hipError_t launch_hvi(const HviArgs &a, hipEvent_t *ev, hipStream_t st);
hipError_t launch_uncertainty(int M, int64_t n, const double *Tm, const double *Em, double *unc,
                              hipEvent_t *ev, hipStream_t st);

struct SelArgs {
    int32_t n_seg;
    int64_t n_cand;
    const int64_t *cand_off, *obs_off, *obs_idx;
    const double *score, *unc;  // unc == nullptr: no exploration pass
    int32_t k[4];               // k1, k2, k3, k
    int npass;                  // 3 or 4
    int64_t max_tiles;          // launch bound on the selection tiles
    int64_t *tile_off;          // [n_seg + 1]
    int32_t *flag;              // [1] set when a score is NaN
    uint64_t *part_key;         // [max_tiles][npass][KR_SEL_LIST]
    int32_t *part_idx;
    int64_t *sel;               // [n_seg][k]
    int32_t *count, *status;
};
hipError_t launch_select(const SelArgs &a, hipEvent_t *ev, hipStream_t st);

// metrics.hip: frontier comparison metrics (Section 6.1).
#define KR_CMP_BLOCKS 512  // blocks of the two reduction passes at most
struct CmpArgs {
    int64_t nA, nB;
    const double *TA, *EA, *TB, *EB;
    int blocks;
    double *part, *part2;  // [blocks][3], [blocks][5]
    double *out;           // [10]
};
hipError_t launch_compare(const CmpArgs &a, hipStream_t st);

// launch_dp.hip: launch-timing frontier of two operation sequences (Appendix B).
struct DpArgs {
    int64_t n_inst;
    int I, J, kmax, out_cap;
    int8_t kind[2 * KR_DP_MAX_OPS];      // S1's kinds, then S2's (1 = communication)
    int8_t run1[KR_DP_MAX_OPS + 1];      // computations in a row from S1[i] (0 at i = I)
    int8_t run2[KR_DP_MAX_OPS + 1];      // the same for S2
    const double *ops;                   // [n_inst][I + J][4]
    double p_static;
    double *out_T, *out_E;               // [n_inst][out_cap]
    int32_t *out_sched;                  // [n_inst][out_cap][I + J] or null
    int32_t *out_n, *status;
    int arena_s, cand_s;                 // first pass's on-chip budget (points, candidates)
    int32_t *retry, *retry_n;            // [2][n_inst], [2]: instances left to larger budgets
};
hipError_t launch_dp(const DpArgs &a, hipStream_t st);

}  // namespace kr
