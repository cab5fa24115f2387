/*
 * kareus.h -- C ABI of the MI355X (gfx950) schedule-search library
 * (libkareus_mi355x.so).
 *
 * Kareus ("Joint Reduction of Dynamic and Static Energy in Large Model Training")
 * plans a training iteration by searching, for every partition, over execution
 * schedules -- the launch position of the communication kernel among the
 * partition's compute kernels, the number of SMs given to communication, and the
 * GPU frequency (Section 4.1) -- keeping each partition's time-energy frontier
 * (Section 4.3, GetFrontier), composing the partition frontiers into the
 * microbatch/iteration frontier (Section 4.4, Algorithm 2) and selecting the
 * schedule behind a frontier point (Section 5.1).  This library runs that search
 * over the whole candidate space with a closed cost model fed by per-kernel time and
 * power tables, on one GPU.  Beside that path it provides:
 *  - the microbatch frontier under Algorithm 2's rules (Section 4.4);
 *  - the scores, batch selection and stopping rule of the multi-pass Bayesian
 *    optimisation (Section 4.3, Algorithm 1);
 *  - the launch-timing frontier of two operation sequences (Appendix B);
 *  - the evaluation's frontier comparison metrics (Section 6.1).
 *
 * Conventions for every entry point
 *  - Array arguments are DEVICE pointers unless marked "host".  The caller owns and
 *    allocates every buffer; the library never allocates or frees device memory and
 *    uses only the workspace the caller passes (size from the matching *_workspace
 *    query).  Workspace contents need no initialisation and are not preserved.
 *  - All work is enqueued on `stream` (a hipStream_t; NULL = the null stream) in
 *    stream order; no entry point synchronises the device.  Results that depend on
 *    device data (counts, status words) are valid once the stream has reached them.
 *  - Return codes report argument errors found on the host and launch errors.  A
 *    condition found on the device (an output capacity exceeded) is reported through
 *    the device-side count/status outputs documented per call.  On any error the
 *    outputs are unspecified but no memory outside the documented extents is written.
 *  - fp64 everywhere; no FMA contraction; every rounding follows the documented
 *    order, so results are reproducible bit for bit across runs and launch shapes.
 *  - Inputs must be finite and non-negative: times, powers, energies (-0.0 counts as 0).
 *    The entry points that take cost tables or point sets accept an optional device
 *    status word (status_out, NULL to skip): when given, a check pass reads every input
 *    value first and the word receives KR_OK, or KR_ENONFINITE if some value is NaN,
 *    infinite or negative (the check reads the inputs once more, so callers that
 *    validated them already pass NULL).  kr_compose_frontiers always checks its points
 *    while it reads them.  With invalid inputs the other outputs are unspecified but
 *    memory-safe.
 */
#ifndef KAREUS_H
#define KAREUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t kr_status;
#define KR_OK 0
#define KR_EINVAL (-1)       /* null pointer, size out of range, inconsistent shape */
#define KR_ENONFINITE (-2)   /* an input time, power or energy is NaN, infinite or negative */
#define KR_ECAPACITY (-3)    /* workspace or output capacity too small (host-known) */
#define KR_EHIP (-4)         /* a HIP runtime call or kernel launch failed */
#define KR_EUNSUPPORTED (-5) /* shape beyond the kernels' on-chip limits */

/*
 * One batch of P partitions and its candidate axes (Sections 4.1-4.2).
 *
 * A partition is one communication kernel stream plus N compute kernels that run in
 * order with no data dependence on it (Section 4.2).  M = 1 or 2 comm kernels run in
 * FIFO order on one comm stream (Section 5.2); the two-kernel form covers the
 * unfused consecutive collectives that Section 4.5 mentions.
 *
 * Candidate axes: frequency index f in [0, F); per comm kernel m a launch position
 * p_m in [0, n_pos) -- the comm kernel is launched together with compute kernel p_m
 * (Section 3.2.2), p_m = N meaning after the last one -- with p_1 <= p_2 when M = 2;
 * and per comm kernel an SM choice s_m in [0, S).
 *
 * Candidate index within a partition (frequency slowest, SM choice fastest):
 *   M = 1: idx = (f * n_pos + p) * S + s
 *   M = 2: pairs (p1 <= p2) ranked lexicographically as pp in [0, n_pos(n_pos+1)/2);
 *          idx = (f * n_pp + pp) * S * S + s1 * S + s2
 */
typedef struct kr_space {
    int32_t n_parts;   /* P >= 1 */
    int32_t n_kernels; /* N >= 1 compute kernels per partition */
    int32_t n_comm;    /* M, 1 or 2 */
    int32_t n_freq;    /* F >= 1 */
    int32_t n_sm;      /* S >= 1 comm SM choices */
    int32_t n_pos;     /* 1 <= n_pos <= N + 1 launch positions */
    double p_static;   /* static power in W (Sections 2.1, 4.5) */
} kr_space;

/*
 * Table layout (row-major fp64, device):
 *   t [P][F][N][S+1]  compute kernel time (s); SM state 0 = no comm running (all SMs),
 *                     state s+1 = comm holds SM choice s (Section 3.2.1)
 *   pw[P][F][N][S+1]  compute kernel dynamic power (W) in that state
 *   tc[P][F][M][S]    comm kernel time (s) with SM choice s
 *   pc[P][F][M][S]    comm kernel dynamic power (W) with SM choice s
 *
 * Cost model (the paper obtains time and energy by profiling and gives no closed
 * form, Section 4.3.1; this is the library's fluid reading of Sections 3.2 and 4.2):
 * compute kernels progress at 1/t in the current SM state and draw pw; comm kernel m
 * is launched when compute reaches the start of kernel p_m, starts when the comm
 * stream is free, runs tc regardless of compute and draws pc; a kernel interrupted
 * by a state change keeps its finished fraction.  Partition time T = the later of
 * compute end and last comm end; energy E = p_static * T + compute dynamic energy +
 * comm dynamic energy (Sections 2.1, 2.3, 4.5).
 */

/*
 * kr_evaluate_partition -- time and energy of every candidate schedule
 * (Section 4.1 decision variables; cost model above).
 *   T_out, E_out  [P][C] with C = F * (n_pos * S) for M = 1, F * (n_pp * S * S) for
 *                 M = 2, indexed by the candidate index above.
 *   status_out    device [1] or NULL: input check (conventions above)
 * Limits: the per-(partition, frequency) table slab staged on chip,
 * 8 * (2N(S+1) + 2(N+1)(S+1) + 2MS) bytes plus 4 bytes per launch-position pair when
 * M = 2, must fit in 64 KiB, else KR_EUNSUPPORTED.  No workspace.
 */
kr_status kr_evaluate_partition(const kr_space *space, const double *t, const double *pw,
                                const double *tc, const double *pc, double *T_out,
                                double *E_out, int32_t *status_out, void *stream);

/* Candidates per partition of `space` (0 if the space is invalid). */
int64_t kr_candidates_per_partition(const kr_space *space);

/*
 * kr_pareto_filter -- GetFrontier per segment (Algorithm 1's return value,
 * Algorithm 2's last step).
 *
 * Segment g holds points [seg_off[g], seg_off[g+1]) of T/E.  A point is kept iff no
 * point of its segment is no worse in time and energy and better in one; among exact
 * (T, E) duplicates the smallest index is kept.  The output per segment is a strict
 * staircase in ascending T (T strictly increasing, E strictly decreasing).
 *   n_total        host; = seg_off[n_seg]
 *   T, E           [n_total] device; finite, >= 0 (-0.0 is read, and reported, as +0.0)
 *   seg_off        device [n_seg + 1]: non-decreasing, seg_off[0] = 0,
 *                  seg_off[n_seg] = n_total, every segment shorter than 2^31 (trusted:
 *                  the host does not read it)
 *   cap            host; capacity of out_idx/out_T/out_E
 *   out_off        device [n_seg + 1]: out_off[g] = start of segment g's frontier;
 *                  out_off[n_seg] = total frontier points, even if > cap
 *   out_idx        device [cap] point index relative to its segment start
 *   out_T, out_E   device [cap]
 *   status_out     device [1] or NULL: input check of T and E (conventions above)
 * If the total exceeds cap, only the first cap points are written; check
 * out_off[n_seg] after the stream completes.
 */
kr_status kr_pareto_filter(int64_t n_total, const double *T, const double *E,
                           const int64_t *seg_off, int32_t n_seg, int64_t cap, int64_t *out_off,
                           int32_t *out_idx, double *out_T, double *out_E, int32_t *status_out,
                           void *ws, size_t ws_bytes, void *stream);
size_t kr_pareto_filter_workspace(int64_t n_total, int32_t n_seg);

/*
 * kr_pareto_filter_noalloc -- kr_pareto_filter for callers that cannot allocate device
 * memory or pass a workspace (code under HIP graph capture, tight serving loops, hosts
 * that forbid allocation): the same call and results, with its workspace in a fixed
 * array inside the library (KR_NOALLOC_SCRATCH_MIB MiB of device memory on each device
 * the call runs on, held until the process ends; nothing is allocated per call).  The
 * caller still passes inputs and outputs.  Limits: n_total <= KR_NOALLOC_MAX_POINTS and
 * n_seg <= KR_NOALLOC_MAX_SEGS, else KR_ECAPACITY before any launch.  Every call on a
 * device shares that device's array: calls that overlap on one device (two streams,
 * two threads) race and must be serialised by the caller.  KR_EHIP if the array's
 * device address cannot be obtained.
 */
#define KR_NOALLOC_MAX_POINTS (1 << 20)
#define KR_NOALLOC_MAX_SEGS (1 << 16)
#define KR_NOALLOC_SCRATCH_MIB 44
kr_status kr_pareto_filter_noalloc(int64_t n_total, const double *T, const double *E,
                                   const int64_t *seg_off, int32_t n_seg, int64_t cap,
                                   int64_t *out_off, int32_t *out_idx, double *out_T,
                                   double *out_E, int32_t *status_out, void *stream);

/*
 * kr_evaluate_and_filter -- kr_evaluate_partition followed by kr_pareto_filter with
 * one segment per partition, fused: candidate T/E never reach device memory, only
 * tile-local frontiers do.  Arguments as in the two calls; out_idx holds candidate
 * indices.  Results are identical to the unfused pair.
 */
kr_status kr_evaluate_and_filter(const kr_space *space, const double *t, const double *pw,
                                 const double *tc, const double *pc, int64_t cap,
                                 int64_t *out_off, int32_t *out_idx, double *out_T,
                                 double *out_E, int32_t *status_out, void *ws, size_t ws_bytes,
                                 void *stream);
size_t kr_evaluate_and_filter_workspace(const kr_space *space);

/*
 * kr_compose_frontiers -- compose partition frontiers into the frontier of their
 * sequential execution (Section 4.4, Algorithm 2), by min-plus convolution over a
 * discretised time axis, plus the non-dominated bins of the result.
 *
 * Partition k's points are [off[k], off[k+1]) of T/E (any finite set with E >= 0,
 * not necessarily sorted or strict; -0.0 energies are binned as +0.0).  With bin width delta, point j of partition k sits
 * at offset off_k[j] = floor((T[j] - tmin_k) / delta); e_k[b] = least E at offset b
 * (ties: smallest point index).  F_1 = e_1 and
 *   F_k[b] = min over b2 of F_{k-1}[b - b2] + e_k[b2]   (ties: smallest b2),
 * so F_P[b] is the least energy of any one-point-per-partition choice whose offsets
 * add up to b, i.e. whose time lies in [tmin_sum + b*delta, tmin_sum + (b+P)*delta).
 * delta = (sum_k range_k) / (n_bins - 1) (1.0 if that sum is 0), nudged up one ulp at
 * a time until 1 + sum_k floor(range_k / delta) <= n_bins; or the caller's delta > 0.
 *
 *   n_parts      host P >= 1; off device [P+1] (every partition non-empty)
 *   n_bins       host B >= 2
 *   F_out        device [B]       F_P (+inf where unreachable)
 *   bp_out       device [P][B]    point index (relative to its partition) chosen for
 *                                 partition k at composite bin b of F_k; -1 if none
 *   bp_off_out   device [P][B] or NULL: the offset of that point (-1 if none), so
 *                                 that a walk back needs one table instead of two
 *   pt_bin_out   device [off[P]]  offset of every point
 *   info_out     device [2]       delta, tmin_sum
 *   L_out        device [1]       reachable bins 1 + sum_k M_k
 *   stair_bin, stair_Tlo, stair_E  device [B]: bins b with F_P[b] below every earlier
 *                                 bin, their lower time edge tmin_sum + b*delta, F_P[b]
 *   n_stair      device [1]       number of staircase bins
 *   status_out   device [1]       KR_OK, or KR_ECAPACITY if the caller's delta needs
 *                                 more than B bins, KR_EINVAL for an empty partition, or
 *                                 KR_ENONFINITE for a non-finite time or an energy that
 *                                 is not a finite value >= 0 (then nothing else is
 *                                 meaningful and n_stair is 0)
 */
kr_status kr_compose_frontiers(int32_t n_parts, const int64_t *off, const double *T,
                               const double *E, int32_t n_bins, double delta, double *F_out,
                               int32_t *bp_out, int32_t *bp_off_out, int32_t *pt_bin_out,
                               double *info_out,
                               int32_t *L_out, int32_t *stair_bin, double *stair_Tlo,
                               double *stair_E, int32_t *n_stair, int32_t *status_out,
                               void *ws, size_t ws_bytes, void *stream);
size_t kr_compose_frontiers_workspace(int32_t n_parts, int32_t n_bins);

/*
 * kr_extract_schedule -- the per-partition choice behind composed bins (schedule
 * selection for a target latency, Section 5.1).  For each query bin, walk the
 * back-pointers from the last partition to the first, peeling off each chosen
 * point's offset.
 *   bp, pt_bin, off, T, E   as produced / consumed by kr_compose_frontiers
 *   bp_off        the offsets kr_compose_frontiers recorded in bp_off_out, or NULL.
 *                 With them the walk reads one table, many rows ahead; without them it
 *                 looks each chosen point's offset up in pt_bin (same results)
 *   bins          device [n_q] query bins
 *   cand_idx      device [off[P]] or NULL: candidate index of every frontier point
 *                 (out_idx of kr_evaluate_and_filter); when given, choice_cand_out
 *                 receives the candidate index of each choice
 *   choice_out    device [n_q][P] point index per partition
 *   choice_cand_out device [n_q][P] or NULL
 *   T_out, E_out  device [n_q] exact sums of the chosen points' T and E, in
 *                 partition order (E equals F_P[bin] bit for bit)
 *   ok_out        device [n_q] 1 if the bin was reachable and the walk consistent
 */
kr_status kr_extract_schedule(int32_t n_parts, int32_t n_bins, const int32_t *bp,
                              const int32_t *bp_off, const int32_t *pt_bin,
                              const int64_t *off, const double *T,
                              const double *E, const int32_t *bins, int32_t n_q,
                              const int32_t *cand_idx, int32_t *choice_out,
                              int32_t *choice_cand_out, double *T_out, double *E_out,
                              int32_t *ok_out, void *stream);

/*
 * kr_microbatch_frontier -- the microbatch frontier of Algorithm 2 with its two rules
 * (Section 4.4): one GPU frequency for the whole microbatch, and one shared SM
 * allocation and launch timing for all partitions of a type; the non-partition
 * components are added per frequency.  A configuration's time is the sum of its
 * partitions' times in execution order, then the components' times at its frequency in
 * their order (energy alike).  Per frequency, the used types are composed as in
 * kr_compose_frontiers with type t's points scaled to (n_t T, n_t E), n_t = its count
 * in seq; each non-dominated bin is walked back to its configuration, whose exact sums
 * enter GetFrontier over all frequencies (ties in order (frequency, bin)).  A frequency
 * at which a used type has no point contributes nothing.
 *   n_types K <= KR_MB_MAX_TYPES, n_freq F      host
 *   seg_off   device [K*F+1]: type t's points at frequency f are seg_off[t*F+f] ..
 *             seg_off[t*F+f+1]-1 of T, E (for instance per-(type, frequency) frontiers
 *             from kr_pareto_filter); n_points host = seg_off[K*F]
 *   n_seq, seq      host [n_seq] type of each partition, in execution order
 *                   (1 <= n_seq <= KR_MB_MAX_SEQ)
 *   n_comp          host >= 0; comp_T, comp_E device [n_comp][F] (NULL when 0)
 *   n_bins          host B >= 2, bins of each frequency's composition
 *   cap             host: capacity of the outputs
 *   out_T, out_E    device [cap] frontier points in ascending time
 *   out_f           device [cap] frequency index of each point
 *   out_choice      device [cap][K] point index within its (type, frequency)
 *                   segment, -1 for types not in seq
 *   n_out           device [1] number of frontier points (the first cap are written)
 * Returns KR_EINVAL for bad arguments (a type out of range in seq, ...), KR_ECAPACITY
 * if ws_bytes is below kr_microbatch_frontier_workspace(...).  Stream-ordered; the host
 * array seq may be reused as soon as the call returns.
 */
#define KR_MB_MAX_TYPES 32
#define KR_MB_MAX_SEQ 2048 /* partitions per microbatch */
size_t kr_microbatch_frontier_workspace(int32_t n_types, int32_t n_freq, int64_t n_points,
                                        int32_t n_seq, int32_t n_bins);
kr_status kr_microbatch_frontier(int32_t n_types, int32_t n_freq, const int64_t *seg_off,
                                 const double *T, const double *E, int64_t n_points,
                                 int32_t n_seq, const int32_t *seq, int32_t n_comp,
                                 const double *comp_T, const double *comp_E, int32_t n_bins,
                                 int64_t cap, double *out_T, double *out_E, int32_t *out_f,
                                 int32_t *out_choice, int64_t *n_out, void *ws, size_t ws_bytes,
                                 void *stream);

/*
 * kr_microbatch_enumerate -- the same microbatch frontier (Section 4.4, Algorithm 2) by
 * enumerating every configuration, as the algorithm is written, with no time grid: for
 * every frequency, every choice of one point per type in seq, summed in execution order
 * and then over the components; GetFrontier over all of them.  Configurations of one
 * frequency are ordered mixed-radix with the first type in seq (in type order) slowest;
 * exact ties go to the order (frequency, that index).  Arguments as for
 * kr_microbatch_frontier, and:
 *   n_configs  host: configurations to reserve, >= the sum over frequencies of the product
 *              of the used types' point counts (<= 2^31 - 1)
 *   status_out device [1]: KR_OK, or KR_ECAPACITY if the configurations exceed n_configs
 *              (then *n_out = 0)
 */
size_t kr_microbatch_enumerate_workspace(int32_t n_types, int32_t n_freq, int64_t n_configs);
kr_status kr_microbatch_enumerate(int32_t n_types, int32_t n_freq, const int64_t *seg_off,
                                  const double *T, const double *E, int32_t n_seq,
                                  const int32_t *seq, int32_t n_comp, const double *comp_T,
                                  const double *comp_E, int64_t n_configs, int64_t cap,
                                  double *out_T, double *out_E, int32_t *out_f,
                                  int32_t *out_choice, int64_t *n_out, int32_t *status_out,
                                  void *ws, size_t ws_bytes, void *stream);

/*
 * kr_hvi_scores -- the three exploitation scores of the multi-pass Bayesian optimisation
 * (Section 4.3, Algorithm 1) for every candidate of every partition: the hypervolume
 * improvement HVI(y) = HV(P u {y}; r) - HV(P; r) of the candidate's predicted point y
 * over the current frontier P, with energy taken as
 *     v = 0 total E,   v = 1 dynamic E - p_static * T,   v = 2 static p_static * T
 * (static energy is static power times time, dynamic is the rest: Sections 2.1, 4.3).
 * For variant v, P is the frontier of the partition's measured points in the
 * (T, energy_v) plane and r = (1.1 * max T, 1.1 * max energy_v) over those points
 * (Appendix C).  HV(S; r) is the area of the part of the box below r that S weakly
 * dominates.
 *   n_seg            host >= 1 partitions
 *   n_cand           host = cand_off[n_seg]; cand_off device [n_seg + 1] non-decreasing
 *                    from 0 (trusted: the host does not read it)
 *   T_hat, E_hat     device [n_cand] predicted time and total energy of each candidate
 *   n_obs            host = obs_off[n_seg]; obs_off device [n_seg + 1] non-decreasing
 *                    from 0, every partition with 1 .. KR_HVI_MAX_OBS measured points
 *   T_obs, E_obs     device [n_obs] measured time and total energy
 *   p_static         host, static power (same unit as energy / time)
 *   hvi_out          device [3][n_cand]: hvi_out[v * n_cand + x]
 *   hv_out           device [n_seg][3]: HV of the measured points per variant (the
 *                    stopping rule's quantity for v = 0)
 *   ref_out          device [n_seg][4]: rT, then rE for v = 0, 1, 2
 *   status_out       device [1]: KR_OK, or KR_EINVAL when a partition has no or more than
 *                    KR_HVI_MAX_OBS measured points (its scores, HV and r are then NaN)
 * HV and r are exact to the oracle's rounding (staircase strips summed in ascending
 * time); HVI is the area y adds, summed strip by strip, so it differs from the
 * difference of two hypervolumes only by rounding (a few ulps of HV(P u {y})).
 * Dominated candidates and candidates outside the box score exactly 0.
 */
#define KR_HVI_MAX_OBS 512
size_t kr_hvi_scores_workspace(int32_t n_seg, int64_t n_obs);
kr_status kr_hvi_scores(int32_t n_seg, int64_t n_cand, const int64_t *cand_off,
                        const double *T_hat, const double *E_hat, int64_t n_obs,
                        const int64_t *obs_off, const double *T_obs, const double *E_obs,
                        double p_static, double *hvi_out, double *hv_out, double *ref_out,
                        int32_t *status_out, void *ws, size_t ws_bytes, void *stream);

/*
 * kr_uncertainty -- the exploration score of Algorithm 1 (Section 4.3): the standard
 * deviation of the ensemble members' predicted time plus that of their predicted
 * energy, per candidate.  Population standard deviation (divide by M); the mean and the
 * squared deviations are summed in member order.
 *   n_members  host M, 1 .. 64
 *   n          host candidates
 *   T_m, E_m   device [M][n] member-major predictions
 *   unc_out    device [n]
 */
kr_status kr_uncertainty(int32_t n_members, int64_t n, const double *T_m, const double *E_m,
                         double *unc_out, void *stream);

/*
 * kr_select_batch -- the multi-pass candidate selection of Algorithm 1 (Section 4.3),
 * per partition g with candidates X (local indices 0 .. n_g - 1) and measured set D:
 *     C = TopK(score_0 over X \ D, k1) u TopK(score_1 over X \ D, k2)
 *         u TopK(score_2 over X \ D, k3)
 *     C = C u TopK(unc over X \ D \ C, k - |C|)           (skipped when unc is NULL)
 * TopK takes the largest scores, ties to the smaller index (all of the set if it is
 * smaller); -0 and +0 tie.  C is written in the order the passes add it (each pass in
 * rank order, members already in C skipped).
 *   n_seg, n_cand, cand_off   as for kr_hvi_scores; every partition < 2^31 candidates
 *   score            device [3][n_cand] (e.g. hvi_out of kr_hvi_scores)
 *   unc              device [n_cand] or NULL
 *   obs_off          device [n_seg + 1]; obs_idx device [obs_off[n_seg]]: the measured
 *                    candidates' local indices (entries outside [0, n_g) are ignored)
 *   k1, k2, k3, k    host: 0 <= k1, k2, k3; k1 + k2 + k3 <= k <= KR_SELECT_MAX_K
 *   sel_out          device [n_seg][k]: the first count_out[g] entries of row g are C
 *   count_out        device [n_seg]
 *   status_out       device [1]: KR_OK, or KR_EINVAL if any score (or unc) is NaN (then
 *                    every count is 0)
 * Selections are exact: the same inputs give the oracle's selection bit for bit.
 */
#define KR_SELECT_MAX_K 64
size_t kr_select_batch_workspace(int32_t n_seg, int64_t n_cand);
kr_status kr_select_batch(int32_t n_seg, int64_t n_cand, const int64_t *cand_off,
                          const double *score, const double *unc, const int64_t *obs_off,
                          const int64_t *obs_idx, int32_t k1, int32_t k2, int32_t k3, int32_t k,
                          int64_t *sel_out, int32_t *count_out, int32_t *status_out, void *ws,
                          size_t ws_bytes, void *stream);

/*
 * kr_hv_converged -- the stopping rule of Algorithm 1 (Appendix C), on the host: after
 * batch b the relative HV improvement is (hv[b] - hv[b-1]) / hv[b-1]; stop once the mean
 * of the last R of them is below eps.  hv_history host [n]: hv[0] after the initial
 * sample, hv[b] after batch b.  A zero hv[b-1] in the window never converges.
 * Returns 1 to stop, 0 to go on (also when fewer than R batches have run or R < 1).
 */
int32_t kr_hv_converged(int32_t n, const double *hv_history, int32_t R, double eps);

/*
 * kr_compare_frontiers -- the evaluation's frontier metrics (Section 6.1, "Metrics") of
 * point set B (a method's frontier) against point set A (the baseline's), in percent
 * of the baseline's value, (base - x) / base * 100:
 *   out[0], out[1]  max-throughput comparison: time and energy reduction of B's
 *                   leftmost point against A's (leftmost = least time, ties to the
 *                   least energy)
 *   out[2]          iso-time energy reduction at the deadline d = A's least time, with
 *                   E_X(d) = least energy among X's points of time <= d
 *   out[3]          iso-energy time reduction at the budget b = A's least energy, with
 *                   T_X(b) = least time among X's points of energy <= b
 *   out[4..6]       d, E_A(d), E_B(d);   out[7..9]  b, T_A(b), T_B(b)
 * A metric is NaN when B has no point within the deadline or budget.  The points may
 * come in any order and include dominated ones.  Every value is exact (minima under
 * predicates) and equals the oracle's bit for bit.
 *   nA, nB            host >= 1
 *   TA, EA / TB, EB   device [nA] / [nB]
 *   out               device [10]
 */
size_t kr_compare_frontiers_workspace(void);
kr_status kr_compare_frontiers(int64_t nA, const double *TA, const double *EA, int64_t nB,
                               const double *TB, const double *EB, double *out, void *ws,
                               size_t ws_bytes, void *stream);

/*
 * kr_launch_timing_frontier -- the launch-timing frontier of two operation sequences by
 * the dynamic program of Appendix B, for a batch of instances that share the sequences'
 * structure (one instance per frequency and SM allocation, say).
 *
 * S1 = ops 0 .. I-1 and S2 = ops I .. I+J-1 each run in order; ops of different
 * sequences are independent.  kind[o] = 0 for a computation, 1 for a communication (a
 * run of consecutive collectives counts as one).  A schedule is a sequence of groups:
 * the next op of S1 alone (code 0), the next op of S2 alone (code 32), S1's next op, a
 * communication, overlapped with S2's next k computations (code 64 + k), or S2's next
 * communication overlapped with S1's next k computations (code 96 + k), k = 1 .. kmax.
 * Groups run one after another.  In an overlapped group both sides start together, the
 * computations run in order with the shared-state time and power until the
 * communication ends and with the alone time and power after it (the partition cost
 * model's fluid progress), and the group ends when both are done.  A group's energy is
 * its dynamic energy plus p_static times its time; a schedule sums its groups.
 * P(i, j) = GetFrontier over the four cases of (group + P(successor)), P(I, J) =
 * {(0, 0)}; exact duplicates keep the first candidate in the order (case, k, the
 * successor's point in ascending time).  Bit-exact with the oracle.
 *   n_inst          host >= 0 instances
 *   I, J            host 0 .. KR_DP_MAX_OPS, I + J >= 1
 *   kind            host [I + J]
 *   ops             device [n_inst][I + J][4]: computation (time alone, power alone,
 *                   time shared, power shared); communication (time, power, -, -)
 *   kmax            host 0 .. KR_DP_MAX_K
 *   out_cap         host 1 .. 64: points kept per instance
 *   out_T, out_E    device [n_inst][out_cap]: P(0, 0) in ascending time
 *   out_sched       device [n_inst][out_cap][I + J] decision codes padded with -1, or
 *                   NULL
 *   out_n           device [n_inst]: frontier size (may exceed out_cap), or -1 when the
 *                   instance exceeded an on-chip limit (a cell frontier above
 *                   KR_DP_CELL_CAP points, more than KR_DP_CAND candidates in a cell, or
 *                   more than KR_DP_ARENA points over all cells)
 *   status_out      device [1]: KR_OK, or KR_ECAPACITY if any instance hit a limit
 * Instances are first solved with a small on-chip budget (many per compute unit); the
 * few that need more are queued and solved again with half the full arena, and the
 * rest with the full budget.
 */
#define KR_DP_MAX_OPS 24
#define KR_DP_MAX_K 16
#define KR_DP_CELL_CAP 64
#define KR_DP_CAND 1024
#define KR_DP_ARENA 2048
size_t kr_launch_timing_frontier_workspace(int64_t n_inst);
kr_status kr_launch_timing_frontier(int64_t n_inst, int32_t I, int32_t J, const int32_t *kind,
                                    const double *ops, double p_static, int32_t kmax,
                                    int32_t out_cap, double *out_T, double *out_E,
                                    int32_t *out_sched, int32_t *out_n, int32_t *status_out,
                                    void *ws, size_t ws_bytes, void *stream);

/*
 * kr_decode_candidates -- candidate index -> (frequency index, launch positions, SM
 * choices) under the index order above.
 *   idx [n] device; f_out [n]; pos_out [n][M]; sm_out [n][M] (device)
 */
kr_status kr_decode_candidates(const kr_space *space, const int32_t *idx, int64_t n,
                               int32_t *f_out, int32_t *pos_out, int32_t *sm_out,
                               void *stream);

/*
 * kr_set_phase_events -- instrumentation for profilers and benchmarks (not part of the
 * method).  When both events are non-NULL, later calls record `start_event` on their
 * stream right before the phase's first kernel and `stop_event` right after its last
 * one; NULL events switch the phase's recording off.  Events are hipEvent_t handles
 * owned by the caller, who must switch the phase off (NULL, NULL) before destroying
 * them.  The setting is per host thread: it applies to later calls made from the
 * thread that set it, and no other thread sees it.
 *   KR_PHASE_EVAL_TILE  the fused evaluation + tile-frontier kernel of
 *                       kr_evaluate_and_filter
 *   KR_PHASE_MERGE      its staircase merges and output compaction
 *   KR_PHASE_MINPLUS    the min-plus steps of kr_compose_frontiers
 *   KR_PHASE_HVI        the per-candidate score kernel of kr_hvi_scores
 *   KR_PHASE_SELECT     the per-tile top-k kernel of kr_select_batch
 *   KR_PHASE_UNC        the kernel of kr_uncertainty
 */
#define KR_PHASE_EVAL_TILE 0
#define KR_PHASE_MERGE 1
#define KR_PHASE_MINPLUS 2
#define KR_PHASE_HVI 3
#define KR_PHASE_SELECT 4
#define KR_PHASE_UNC 5
kr_status kr_set_phase_events(int32_t phase, void *start_event, void *stop_event);

/* Human-readable name of a status code. */
const char *kr_status_string(kr_status status);

#ifdef __cplusplus
}
#endif

#endif /* KAREUS_H */
