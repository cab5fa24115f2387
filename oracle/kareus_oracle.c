/*
 * Kareus schedule-search hot path: CPU ORACLE.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or load this
 * file; only the tests, the smoke check and the benchmark's CPU-baseline leg use it.
 * It is plain, slow and single-threaded on purpose, and shares no code, header, table
 * or helper with the HIP library.  Build: gcc -O2 -ffp-contract=off -fPIC -shared.
 *
 * What it computes (Kareus, "Joint Reduction of Dynamic and Static Energy in Large
 * Model Training"):
 *   oracle_evaluate   time and energy of every candidate execution schedule of one
 *                     partition (Sections 4.1-4.2; energy model of Sections 2.1, 2.3,
 *                     4.3.2 and 4.5).  The paper gives no closed-form cost model
 *                     (Section 4.3.1 says time and energy come from profiling), so
 *                     this follows a fluid SM-share reading written out below.
 *   oracle_pareto     GetFrontier: the non-dominated (time, energy) set (Algorithm 1's
 *                     return value; Algorithm 2's last step).
 *   oracle_compose    partition frontiers -> summed (time, energy) over every choice
 *                     of one point per partition, pruned to a frontier (Section 4.4,
 *                     Algorithm 2), done as a min-plus recurrence over a discretised
 *                     time axis.
 *   oracle_staircase  the non-dominated points of the composed array.
 *   oracle_extract    the per-partition choice behind a composed point (schedule
 *                     selection for a target latency, Section 5.1).
 *   oracle_microbatch the microbatch frontier of Algorithm 2 with its two rules: one
 *                     GPU frequency for the whole microbatch, and one shared SM
 *                     allocation and launch timing per partition type (Section 4.4),
 *                     plus the non-partition components, composed on a time grid.
 *   oracle_microbatch_exact  the same frontier by enumerating every configuration, as
 *                     Algorithm 2 is written.
 *   oracle_hypervolume, oracle_hvi, oracle_uncertainty, oracle_select,
 *   oracle_hv_converged  the scores, candidate selection and stopping rule of the
 *                     multi-pass Bayesian optimisation (Section 4.3, Algorithm 1,
 *                     Appendix C).
 *   oracle_compare    the evaluation's frontier metrics: max-throughput, iso-time
 *                     energy and iso-energy time reductions (Section 6.1).
 *   oracle_launch_dp  the launch-timing frontier of two operation sequences by the
 *                     dynamic program of Appendix B.
 *
 * Every floating-point line is one IEEE fp64 rounding in the written order; the file
 * must be compiled without FMA contraction and without fast-math.
 */
#define _GNU_SOURCE /* qsort_r: reentrant sorts, so partitions may run on threads */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_EINVAL -1
#define OR_ECAPACITY -3

/* ------------------------------------------------------------------------------
 * Cost model of one partition (Sections 3.2 and 4.2).
 *
 * A partition holds N compute kernels that run in order on the compute stream and M
 * (1 or 2) communication kernels with no data dependence on them (Section 4.2).  A
 * candidate fixes the GPU frequency f, and for each comm kernel m its launch
 * position p_m and SM choice s_m (Section 4.1).
 *
 * Readings (the paper is silent; Sections 4.3.1 and Appendix B):
 *  - launch position p means the comm kernel is launched together with compute
 *    kernel p, i.e. when compute reaches the start of kernel p; p = N launches it
 *    after the last compute kernel (fully exposed) (Section 3.2.2).
 *  - SMs given to communication are taken from compute (Section 3.2.1): while comm m
 *    runs, compute runs in SM state sigma_m = s_m + 1, whose per-kernel time and
 *    power come from the tables; otherwise it runs in state 0 (all SMs).
 *  - progress is fluid: a kernel interrupted by a state change keeps the finished
 *    fraction of its work.
 *  - comm kernels share one comm stream in FIFO order (Section 5.2: compute and comm
 *    on separate streams, events for launch timing); comm m starts at the later of
 *    its launch and the end of comm m-1, and runs for tc regardless of compute.
 *  - energy = static power x partition time + dynamic energy of compute and comm
 *    (Sections 2.1, 2.3 and 4.5); idle compute draws no dynamic power; the
 *    partition ends when both compute and the last comm kernel have finished.
 * ---------------------------------------------------------------------------- */

typedef struct {
    int N;            /* compute kernels */
    int S1;           /* SM states = S + 1 */
    const double *t;  /* [N][S1] kernel time in each state, this frequency */
    const double *pw; /* [N][S1] kernel dynamic power in each state */
    const double *A;  /* [S1][N+1] A[s][i] = sum_{j<i} t[j][s], left to right */
    const double *B;  /* [S1][N+1] B[s][i] = sum_{j<i} pw[j][s]*t[j][s] */
    int i;            /* kernel in progress (or next to start) */
    double w;         /* unfinished fraction of kernel i (1.0 = not started) */
    double Ec;        /* compute dynamic energy so far */
} walk_state;

#define TT(W, j, s) ((W)->t[(size_t)(j) * (W)->S1 + (s)])
#define PW(W, j, s) ((W)->pw[(size_t)(j) * (W)->S1 + (s)])
#define AA(W, s, j) ((W)->A[(size_t)(s) * ((W)->N + 1) + (j)])
#define BB(W, s, j) ((W)->B[(size_t)(s) * ((W)->N + 1) + (j)])

/* Run compute in SM state s for at most `budget` seconds or until it reaches the
 * start of kernel `stop` (i <= stop <= N).  Sets *elapsed; returns 1 if `stop` was
 * reached, 0 if the budget ran out first. */
static int run_compute(walk_state *W, int s, double budget, int stop, double *elapsed)
{
    double used = 0.0;
    if (W->w < 1.0) {
        /* finish the interrupted kernel first */
        double need = W->w * TT(W, W->i, s);
        if (need <= budget) {
            W->Ec = W->Ec + PW(W, W->i, s) * need;
            used = need;
            W->i = W->i + 1;
            W->w = 1.0;
        } else {
            W->Ec = W->Ec + PW(W, W->i, s) * budget;
            W->w = W->w - budget / TT(W, W->i, s);
            if (W->w < 0.0) W->w = 0.0;
            *elapsed = budget;
            return 0;
        }
    }
    double rb = budget - used;
    /* whole kernels that fit: the largest j in [i, stop] with A[j] - A[i] <= rb */
    int i0 = W->i;
    int j = i0;
    while (j < stop && (AA(W, s, j + 1) - AA(W, s, i0)) <= rb) j = j + 1;
    W->Ec = W->Ec + (BB(W, s, j) - BB(W, s, i0));
    if (j == stop) {
        *elapsed = used + (AA(W, s, j) - AA(W, s, i0));
        W->i = j;
        return 1;
    }
    /* budget ends inside kernel j */
    double r = rb - (AA(W, s, j) - AA(W, s, i0));
    W->Ec = W->Ec + PW(W, j, s) * r;
    W->w = 1.0 - r / TT(W, j, s);
    if (W->w < 0.0) W->w = 0.0;
    W->i = j;
    *elapsed = budget;
    return 0;
}

/* Time and energy of one candidate at one frequency.
 * tcm, pcm: comm time and power of each comm kernel under its SM choice. */
static void cost_one(walk_state *W, int M, const int *pos, const int *sigma,
                     const double *tcm, const double *pcm, double p_static,
                     double *T_out, double *E_out)
{
    double tau = 0.0, el = 0.0, T = 0.0;
    int m, done = 0;
    W->i = 0;
    W->w = 1.0;
    W->Ec = 0.0;
    for (m = 0; m < M; m++) {
        if (W->i < pos[m]) { /* compute has not yet reached the launch point */
            run_compute(W, 0, INFINITY, pos[m], &el);
            tau = tau + el;
        }
        double start = tau; /* FIFO: tau is also the end of comm m-1 */
        if (run_compute(W, sigma[m], tcm[m], W->N, &el)) {
            /* compute finished while comm m ran; later comm kernels follow it */
            T = start + tcm[m];
            for (int q = m + 1; q < M; q++) T = T + tcm[q];
            done = 1;
            break;
        }
        tau = start + tcm[m];
    }
    if (!done) {
        run_compute(W, 0, INFINITY, W->N, &el);
        T = tau + el;
    }
    double E = p_static * T;
    E = E + W->Ec;
    for (m = 0; m < M; m++) E = E + pcm[m] * tcm[m];
    *T_out = T;
    *E_out = E;
}

/* Candidate index (frequency slowest, SM choice fastest):
 *   M = 1: idx = (f * n_pos + p) * S + s
 *   M = 2: pairs p1 <= p2 ranked lexicographically as pp;
 *          idx = (f * n_pp + pp) * S * S + s1 * S + s2
 * One partition; t, pw: [F][N][S+1]; tc, pc: [F][M][S]; T_out, E_out: [n_cand]. */
int oracle_evaluate(int N, int M, int F, int S, int n_pos, double p_static,
                    const double *t, const double *pw, const double *tc, const double *pc,
                    double *T_out, double *E_out)
{
    if (N < 1 || (M != 1 && M != 2) || F < 1 || S < 1 || n_pos < 1 || n_pos > N + 1)
        return OR_EINVAL;
    int S1 = S + 1;
    double *A = (double *)malloc(sizeof(double) * (size_t)S1 * (N + 1));
    double *B = (double *)malloc(sizeof(double) * (size_t)S1 * (N + 1));
    if (!A || !B) { free(A); free(B); return OR_EINVAL; }
    long long idx = 0;
    for (int f = 0; f < F; f++) {
        const double *tf = t + (size_t)f * N * S1;
        const double *pwf = pw + (size_t)f * N * S1;
        const double *tcf = tc + (size_t)f * M * S;
        const double *pcf = pc + (size_t)f * M * S;
        for (int s = 0; s < S1; s++) {
            A[(size_t)s * (N + 1)] = 0.0;
            B[(size_t)s * (N + 1)] = 0.0;
            for (int i = 0; i < N; i++) {
                double ti = tf[(size_t)i * S1 + s];
                A[(size_t)s * (N + 1) + i + 1] = A[(size_t)s * (N + 1) + i] + ti;
                B[(size_t)s * (N + 1) + i + 1] =
                    B[(size_t)s * (N + 1) + i] + (pwf[(size_t)i * S1 + s] * ti);
            }
        }
        walk_state W = {N, S1, tf, pwf, A, B, 0, 1.0, 0.0};
        int pos[2], sig[2];
        double tcm[2], pcm[2];
        if (M == 1) {
            for (int p = 0; p < n_pos; p++)
                for (int s = 0; s < S; s++) {
                    pos[0] = p;
                    sig[0] = s + 1;
                    tcm[0] = tcf[s];
                    pcm[0] = pcf[s];
                    cost_one(&W, 1, pos, sig, tcm, pcm, p_static, &T_out[idx], &E_out[idx]);
                    idx++;
                }
        } else {
            for (int p1 = 0; p1 < n_pos; p1++)
                for (int p2 = p1; p2 < n_pos; p2++)
                    for (int s1 = 0; s1 < S; s1++)
                        for (int s2 = 0; s2 < S; s2++) {
                            pos[0] = p1;
                            pos[1] = p2;
                            sig[0] = s1 + 1;
                            sig[1] = s2 + 1;
                            tcm[0] = tcf[s1];
                            pcm[0] = pcf[s1];
                            tcm[1] = tcf[S + s2];
                            pcm[1] = pcf[S + s2];
                            cost_one(&W, 2, pos, sig, tcm, pcm, p_static, &T_out[idx],
                                     &E_out[idx]);
                            idx++;
                        }
        }
    }
    free(A);
    free(B);
    return OR_OK;
}

/* ------------------------------------------------------------------------------
 * GetFrontier (Algorithm 1's return value, Algorithm 2's last step).
 * A point is kept iff no other point is at least as good in both time and energy
 * and strictly better in one; of exact (time, energy) duplicates the smallest index
 * is kept.  Done as: sort by (T, E, index), keep a point iff its energy is strictly
 * below every energy before it.  Output is in ascending time.
 * ---------------------------------------------------------------------------- */
typedef struct { const double *T, *E; } te_ctx;

static int cmp_tei(const void *a, const void *b, void *ctx)
{
    const te_ctx *c = (const te_ctx *)ctx;
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    if (c->T[x] < c->T[y]) return -1;
    if (c->T[x] > c->T[y]) return 1;
    if (c->E[x] < c->E[y]) return -1;
    if (c->E[x] > c->E[y]) return 1;
    return (x > y) - (x < y);
}

int oracle_pareto(int64_t n, const double *T, const double *E, int32_t *out_idx, int64_t *n_out)
{
    if (n < 0) return OR_EINVAL;
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    if (!order) return OR_EINVAL;
    for (int64_t k = 0; k < n; k++) order[k] = (int32_t)k;
    te_ctx ctx = {T, E};
    qsort_r(order, (size_t)n, sizeof(int32_t), cmp_tei, &ctx);
    double best = INFINITY;
    int64_t kept = 0;
    for (int64_t k = 0; k < n; k++) {
        int32_t c = order[k];
        if (E[c] < best) {
            out_idx[kept++] = c;
            best = E[c];
        }
    }
    *n_out = kept;
    free(order);
    return OR_OK;
}

/* ------------------------------------------------------------------------------
 * Composition of partition frontiers (Section 4.4, Algorithm 2).
 *
 * The microbatch runs its partitions one after another, so one choice per partition
 * gives time = sum of times and energy = sum of energies; the composed frontier is
 * GetFrontier over every such combination.  Instead of enumerating the Cartesian
 * product, time is discretised: with bin width delta, point j of partition k sits at
 * offset off_k[j] = floor((T_k[j] - tmin_k) / delta), and
 *     F_1[b] = e_1[b],   F_k[b] = min_{b2} F_{k-1}[b - b2] + e_k[b2]
 * where e_k[b2] is the least energy among partition k's points at offset b2.  F_P[b]
 * is the least total energy of any combination whose offsets add up to b, i.e. whose
 * time lies in [tmin_sum + b*delta, tmin_sum + (b+P)*delta).
 *
 * Readings: delta = (sum_k (tmax_k - tmin_k)) / (B - 1) (1.0 if that sum is 0), or
 * the caller's delta > 0; with an automatic delta it is nudged up one ulp at a time
 * until 1 + sum_k floor(range_k / delta) <= B.  Ties in e_k go to the smallest point
 * index; ties in the min-plus go to the smallest b2.
 *
 * off [P+1] point offsets; T, E [off[P]] points; F_out [B]; bp_out [P][B] point
 * index chosen for partition k at composite bin b (-1 = unreachable); pt_bin_out
 * [off[P]] the offset of every point; info_out[0] = delta, info_out[1] = tmin_sum;
 * L_out = number of bins reachable (1 + sum_k M_k).
 * ---------------------------------------------------------------------------- */
int oracle_compose(int P, const int64_t *off, const double *T, const double *E, int B,
                   double delta_in, double *F_out, int32_t *bp_out, int32_t *pt_bin_out,
                   double *info_out, int32_t *L_out)
{
    if (P < 1 || B < 2) return OR_EINVAL;
    for (int k = 0; k < P; k++)
        if (off[k + 1] <= off[k]) return OR_EINVAL;
    double *tmin = (double *)malloc(sizeof(double) * P);
    double *range = (double *)malloc(sizeof(double) * P);
    int64_t *Mk = (int64_t *)malloc(sizeof(int64_t) * P);
    double *e = (double *)malloc(sizeof(double) * (size_t)B);
    int32_t *arg = (int32_t *)malloc(sizeof(int32_t) * (size_t)B);
    double *Fprev = (double *)malloc(sizeof(double) * (size_t)B);
    double *Fcur = (double *)malloc(sizeof(double) * (size_t)B);
    int rc = OR_OK;
    if (!tmin || !range || !Mk || !e || !arg || !Fprev || !Fcur) { rc = OR_EINVAL; goto done; }

    /* 1. per-partition time range */
    for (int k = 0; k < P; k++) {
        double lo = T[off[k]], hi = T[off[k]];
        for (int64_t j = off[k]; j < off[k + 1]; j++) {
            if (T[j] < lo) lo = T[j];
            if (T[j] > hi) hi = T[j];
        }
        tmin[k] = lo;
        range[k] = hi - lo;
    }
    /* 2-3. bin width and per-partition bin counts */
    double R = 0.0;
    for (int k = 0; k < P; k++) R = R + range[k];
    double delta;
    if (delta_in > 0.0) delta = delta_in;
    else if (R > 0.0) delta = R / (double)(B - 1);
    else delta = 1.0;
    for (;;) {
        int64_t total = 1;
        for (int k = 0; k < P; k++) {
            Mk[k] = (int64_t)floor(range[k] / delta);
            total += Mk[k];
        }
        if (total <= B) break;
        if (delta_in > 0.0) { rc = OR_ECAPACITY; goto done; }
        delta = nextafter(delta, INFINITY);
    }
    double tmin_sum = 0.0;
    for (int k = 0; k < P; k++) tmin_sum = tmin_sum + tmin[k];

    /* 4. offsets of every point */
    for (int k = 0; k < P; k++)
        for (int64_t j = off[k]; j < off[k + 1]; j++) {
            int64_t o = (int64_t)floor((T[j] - tmin[k]) / delta);
            if (o > Mk[k]) o = Mk[k];
            pt_bin_out[j] = (int32_t)o;
        }

    for (int64_t x = 0; x < (int64_t)P * B; x++) bp_out[x] = -1;
    int64_t L = 0;
    for (int k = 0; k < P; k++) {
        /* 5. least energy per offset of partition k (ties: smallest point index) */
        for (int64_t b = 0; b <= Mk[k]; b++) {
            e[b] = INFINITY;
            arg[b] = -1;
        }
        for (int64_t j = off[k]; j < off[k + 1]; j++) {
            int32_t b = pt_bin_out[j];
            if (E[j] < e[b]) {
                e[b] = E[j];
                arg[b] = (int32_t)(j - off[k]);
            }
        }
        int32_t *bpk = bp_out + (size_t)k * B;
        if (k == 0) {
            /* 6. F_1 = e_1 */
            L = Mk[0] + 1;
            for (int64_t b = 0; b < B; b++) Fcur[b] = INFINITY;
            for (int64_t b = 0; b < L; b++) {
                Fcur[b] = e[b];
                bpk[b] = arg[b];
            }
        } else {
            /* 7. min-plus step, plain double loop */
            int64_t Lnew = L + Mk[k];
            for (int64_t b = 0; b < B; b++) Fcur[b] = INFINITY;
            for (int64_t b = 0; b < Lnew; b++) {
                double best = INFINITY;
                int32_t who = -1;
                for (int64_t b2 = 0; b2 <= Mk[k]; b2++) {
                    int64_t a = b - b2;
                    if (a < 0 || a >= L) continue;
                    if (!(Fprev[a] < INFINITY) || !(e[b2] < INFINITY)) continue;
                    double v = Fprev[a] + e[b2];
                    if (v < best) {
                        best = v;
                        who = arg[b2];
                    }
                }
                Fcur[b] = best;
                bpk[b] = who;
            }
            L = Lnew;
        }
        double *sw = Fprev;
        Fprev = Fcur;
        Fcur = sw;
    }
    memcpy(F_out, Fprev, sizeof(double) * (size_t)B);
    info_out[0] = delta;
    info_out[1] = tmin_sum;
    *L_out = (int32_t)L;
done:
    free(tmin);
    free(range);
    free(Mk);
    free(e);
    free(arg);
    free(Fprev);
    free(Fcur);
    return rc;
}

/* Non-dominated bins of the composed array: keep b iff F[b] is strictly below every
 * F[b'] with b' < b.  The lower time edge of bin b is tmin_sum + b * delta. */
int oracle_staircase(int B, const double *F, double delta, double tmin_sum,
                     int32_t *bins_out, double *Tlo_out, double *E_out, int32_t *n_out)
{
    double best = INFINITY;
    int32_t n = 0;
    for (int b = 0; b < B; b++)
        if (F[b] < best) {
            best = F[b];
            bins_out[n] = b;
            Tlo_out[n] = tmin_sum + (double)b * delta;
            E_out[n] = F[b];
            n++;
        }
    *n_out = n;
    return OR_OK;
}

/* The per-partition choice behind composite bin `bin`: walk the back-pointers from
 * the last partition to the first, peeling off each chosen point's offset.  Writes
 * the point index per partition, and the exact time and energy of that schedule,
 * summed over partitions in order.  Returns OR_EINVAL if `bin` is unreachable. */
int oracle_extract(int P, int B, const int64_t *off, const double *T, const double *E,
                   const int32_t *bp, const int32_t *pt_bin, int32_t bin,
                   int32_t *choice_out, double *T_out, double *E_out)
{
    if (bin < 0 || bin >= B) return OR_EINVAL;
    int32_t b = bin;
    for (int k = P - 1; k >= 0; k--) {
        int32_t j = bp[(size_t)k * B + b];
        if (j < 0) return OR_EINVAL;
        choice_out[k] = j;
        b = b - pt_bin[off[k] + j];
        if (b < 0) return OR_EINVAL;
    }
    if (b != 0) return OR_EINVAL;
    double Ts = 0.0, Es = 0.0;
    for (int k = 0; k < P; k++) {
        Ts = Ts + T[off[k] + choice_out[k]];
        Es = Es + E[off[k] + choice_out[k]];
    }
    *T_out = Ts;
    *E_out = Es;
    return OR_OK;
}

/* ------------------------------------------------------------------------------
 * Microbatch frontier (Section 4.4, Algorithm 2).
 *
 * A microbatch runs n_seq partitions in order; partition i is of type seq[i].  For a
 * GPU frequency f, every partition of type t uses the same (SM allocation, launch
 * timing) choice, so a configuration is one point of each type's frontier at f.  Its
 * time is the sum of its partitions' times in execution order followed by the
 * non-partition components' times at f (likewise energy); the microbatch frontier is
 * GetFrontier over every configuration of every frequency.
 *
 * Per frequency the configurations are composed on a discretised time axis as in
 * oracle_compose: type t, used n_t > 0 times, contributes its points scaled to
 * (n_t * T, n_t * E) (one rounding each), and the used types are composed in type
 * order.  Every non-dominated bin of that composition (oracle_staircase) is walked
 * back to its choice (oracle_extract); that configuration's time and energy are then
 * summed exactly in execution order, components last.  The union over frequencies of
 * these configurations, in order (frequency, staircase bin), goes through GetFrontier.
 * A frequency at which some used type has no point contributes nothing.
 *
 * seg_off [K*F+1]: points of type t at frequency f are seg_off[t*F+f] ..
 * seg_off[t*F+f+1]-1 of T, E (each such segment a frontier or any point set).
 * cT, cE [n_comp][F].  Outputs up to cap points in ascending time: oT, oE, of
 * (frequency), ochoice [cap][K] (point index within its (type, f) segment; -1 for
 * unused types); *n_out = number of frontier points (may exceed cap).
 * ---------------------------------------------------------------------------- */
int oracle_microbatch(int K, int F, const int64_t *seg_off, const double *T, const double *E,
                      int n_seq, const int32_t *seq, int n_comp, const double *cT,
                      const double *cE, int B, int64_t cap, double *oT, double *oE,
                      int32_t *of, int32_t *ochoice, int64_t *n_out)
{
    if (K < 1 || F < 1 || n_seq < 1 || n_comp < 0 || B < 2 || cap < 0) return OR_EINVAL;
    int32_t *cnt = (int32_t *)calloc((size_t)K, sizeof(int32_t));
    int32_t *used = (int32_t *)malloc(sizeof(int32_t) * (size_t)K);
    if (!cnt || !used) { free(cnt); free(used); return OR_EINVAL; }
    for (int i = 0; i < n_seq; i++) {
        if (seq[i] < 0 || seq[i] >= K) { free(cnt); free(used); return OR_EINVAL; }
        cnt[seq[i]]++;
    }
    int Ku = 0;
    for (int t = 0; t < K; t++)
        if (cnt[t] > 0) used[Ku++] = t;
    int64_t maxpts = 0;
    for (int t = 0; t < K; t++)
        for (int f = 0; f < F; f++) {
            int64_t n = seg_off[t * F + f + 1] - seg_off[t * F + f];
            if (n < 0) { free(cnt); free(used); return OR_EINVAL; }
            if (n > maxpts) maxpts = n;
        }
    int64_t ncand_cap = (int64_t)F * B;
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(Ku + 1));
    double *Ts = (double *)malloc(sizeof(double) * (size_t)(Ku * maxpts + 1));
    double *Es = (double *)malloc(sizeof(double) * (size_t)(Ku * maxpts + 1));
    double *Fb = (double *)malloc(sizeof(double) * (size_t)B);
    int32_t *bp = (int32_t *)malloc(sizeof(int32_t) * (size_t)Ku * B);
    int32_t *pt = (int32_t *)malloc(sizeof(int32_t) * (size_t)(Ku * maxpts + 1));
    int32_t *sb = (int32_t *)malloc(sizeof(int32_t) * (size_t)B);
    double *stl = (double *)malloc(sizeof(double) * (size_t)B);
    double *se = (double *)malloc(sizeof(double) * (size_t)B);
    int32_t *ch = (int32_t *)malloc(sizeof(int32_t) * (size_t)(Ku + 1));
    double *cTm = (double *)malloc(sizeof(double) * (size_t)ncand_cap);
    double *cEm = (double *)malloc(sizeof(double) * (size_t)ncand_cap);
    int32_t *cf = (int32_t *)malloc(sizeof(int32_t) * (size_t)ncand_cap);
    int32_t *cch = (int32_t *)malloc(sizeof(int32_t) * (size_t)ncand_cap * K);
    int32_t *keep = (int32_t *)malloc(sizeof(int32_t) * (size_t)(ncand_cap + 1));
    int rc = OR_OK;
    int64_t nc = 0;
    if (!off || !Ts || !Es || !Fb || !bp || !pt || !sb || !stl || !se || !ch || !cTm || !cEm ||
        !cf || !cch || !keep) {
        rc = OR_EINVAL;
        goto done;
    }
    for (int f = 0; f < F; f++) {
        /* scaled points of the used types, in type order */
        int64_t w = 0;
        int empty = 0;
        off[0] = 0;
        for (int u = 0; u < Ku; u++) {
            int t = used[u];
            int64_t lo = seg_off[t * F + f], hi = seg_off[t * F + f + 1];
            if (hi <= lo) empty = 1;
            for (int64_t j = lo; j < hi; j++) {
                Ts[w] = (double)cnt[t] * T[j];
                Es[w] = (double)cnt[t] * E[j];
                w++;
            }
            off[u + 1] = w;
        }
        if (empty) continue;
        double info[2];
        int32_t L;
        rc = oracle_compose(Ku, off, Ts, Es, B, 0.0, Fb, bp, pt, info, &L);
        if (rc != OR_OK) goto done;
        int32_t ns = 0;
        oracle_staircase(B, Fb, info[0], info[1], sb, stl, se, &ns);
        for (int32_t q = 0; q < ns; q++) {
            double tsum, esum;
            rc = oracle_extract(Ku, B, off, Ts, Es, bp, pt, sb[q], ch, &tsum, &esum);
            if (rc != OR_OK) goto done;
            /* exact time and energy: partitions in execution order, then components */
            double Tm = 0.0, Em = 0.0;
            for (int i = 0; i < n_seq; i++) {
                int t = seq[i], u = 0;
                while (used[u] != t) u++;
                int64_t x = seg_off[t * F + f] + ch[u];
                Tm = Tm + T[x];
                Em = Em + E[x];
            }
            for (int c = 0; c < n_comp; c++) {
                Tm = Tm + cT[(int64_t)c * F + f];
                Em = Em + cE[(int64_t)c * F + f];
            }
            cTm[nc] = Tm;
            cEm[nc] = Em;
            cf[nc] = f;
            for (int t = 0; t < K; t++) cch[nc * K + t] = -1;
            for (int u = 0; u < Ku; u++) cch[nc * K + used[u]] = ch[u];
            nc++;
        }
    }
    {
        int64_t nk = 0;
        rc = oracle_pareto(nc, cTm, cEm, keep, &nk);
        if (rc != OR_OK) goto done;
        for (int64_t r = 0; r < nk && r < cap; r++) {
            int32_t c = keep[r];
            oT[r] = cTm[c];
            oE[r] = cEm[c];
            of[r] = cf[c];
            for (int t = 0; t < K; t++) ochoice[r * K + t] = cch[(int64_t)c * K + t];
        }
        *n_out = nk;
    }
done:
    free(cnt); free(used); free(off); free(Ts); free(Es); free(Fb); free(bp); free(pt);
    free(sb); free(stl); free(se); free(ch); free(cTm); free(cEm); free(cf); free(cch);
    free(keep);
    return rc;
}

/* ------------------------------------------------------------------------------
 * Microbatch frontier by enumeration (Section 4.4, Algorithm 2 as written): for every
 * frequency f, every configuration (one point of each used type's set at f), its time
 * and energy summed in execution order and then over the components, and GetFrontier
 * over all of them.  Configurations of one frequency are taken in mixed-radix order
 * with the first used type (in type order) slowest; the union is in order (f, that
 * index), which decides exact ties.  Same arguments and outputs as oracle_microbatch.
 * ---------------------------------------------------------------------------- */
int oracle_microbatch_exact(int K, int F, const int64_t *seg_off, const double *T,
                            const double *E, int n_seq, const int32_t *seq, int n_comp,
                            const double *cT, const double *cE, int64_t cap, double *oT,
                            double *oE, int32_t *of, int32_t *ochoice, int64_t *n_out)
{
    if (K < 1 || F < 1 || n_seq < 1 || n_comp < 0 || cap < 0) return OR_EINVAL;
    int32_t cnt[64], used[64];
    if (K > 64) return OR_EINVAL;
    for (int t = 0; t < K; t++) cnt[t] = 0;
    for (int i = 0; i < n_seq; i++) {
        if (seq[i] < 0 || seq[i] >= K) return OR_EINVAL;
        cnt[seq[i]]++;
    }
    int Ku = 0;
    for (int t = 0; t < K; t++)
        if (cnt[t] > 0) used[Ku++] = t;
    int64_t total = 0;
    for (int f = 0; f < F; f++) {
        int64_t n = 1;
        for (int u = 0; u < Ku; u++) n *= seg_off[used[u] * F + f + 1] - seg_off[used[u] * F + f];
        total += n;
    }
    double *cTm = (double *)malloc(sizeof(double) * (size_t)(total + 1));
    double *cEm = (double *)malloc(sizeof(double) * (size_t)(total + 1));
    int32_t *cf = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total + 1));
    int32_t *cch = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total + 1) * K);
    int32_t *keep = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total + 1));
    int rc = OR_OK;
    if (!cTm || !cEm || !cf || !cch || !keep) { rc = OR_EINVAL; goto done; }
    {
        int64_t nc = 0;
        int32_t j[64];
        for (int f = 0; f < F; f++) {
            int64_t n = 1;
            for (int u = 0; u < Ku; u++)
                n *= seg_off[used[u] * F + f + 1] - seg_off[used[u] * F + f];
            for (int u = 0; u < Ku; u++) j[u] = 0;
            for (int64_t c = 0; c < n; c++) {
                double Tm = 0.0, Em = 0.0;
                for (int i = 0; i < n_seq; i++) {
                    int u = 0;
                    while (used[u] != seq[i]) u++;
                    int64_t x = seg_off[used[u] * F + f] + j[u];
                    Tm = Tm + T[x];
                    Em = Em + E[x];
                }
                for (int k = 0; k < n_comp; k++) {
                    Tm = Tm + cT[(int64_t)k * F + f];
                    Em = Em + cE[(int64_t)k * F + f];
                }
                cTm[nc] = Tm;
                cEm[nc] = Em;
                cf[nc] = f;
                for (int t = 0; t < K; t++) cch[nc * K + t] = -1;
                for (int u = 0; u < Ku; u++) cch[nc * K + used[u]] = j[u];
                nc++;
                /* next configuration: the last used type fastest */
                for (int u = Ku - 1; u >= 0; u--) {
                    if (++j[u] < seg_off[used[u] * F + f + 1] - seg_off[used[u] * F + f]) break;
                    j[u] = 0;
                }
            }
        }
        int64_t nk = 0;
        rc = oracle_pareto(nc, cTm, cEm, keep, &nk);
        if (rc != OR_OK) goto done;
        for (int64_t r = 0; r < nk && r < cap; r++) {
            int32_t c = keep[r];
            oT[r] = cTm[c];
            oE[r] = cEm[c];
            of[r] = cf[c];
            for (int t = 0; t < K; t++) ochoice[r * K + t] = cch[(int64_t)c * K + t];
        }
        *n_out = nk;
    }
done:
    free(cTm); free(cEm); free(cf); free(cch); free(keep);
    return rc;
}

/* ------------------------------------------------------------------------------
 * Hypervolume and hypervolume improvement (Section 4.3, exploitation passes of
 * Algorithm 1; reference point from Appendix C).
 *
 * HV(S; r) is the area of the part of the box below r = (rT, rE) that some point of S
 * weakly dominates, i.e. the area of the union over s in S of [s.T, rT] x [s.E, rE]
 * (empty unless s.T < rT and s.E < rE).  Measured in vertical strips: visit the
 * points in ascending (T, E); a point inside the box whose energy is below every
 * energy seen so far opens a new step of the staircase, and the previous step's strip
 * (this T - previous T) * (rE - previous E) is added; the last step's strip ends at
 * rT.  The strips are added in ascending time.
 *
 * HVI(y) = HV(S u {y}; r) - HV(S; r), both computed as above.
 * ---------------------------------------------------------------------------- */
typedef struct { double t, e; } or_pt;

static int cmp_pt(const void *a, const void *b)
{
    const or_pt *x = (const or_pt *)a, *y = (const or_pt *)b;
    if (x->t < y->t) return -1;
    if (x->t > y->t) return 1;
    if (x->e < y->e) return -1;
    if (x->e > y->e) return 1;
    return 0;
}

/* pts is sorted in place. */
static double hv_of(or_pt *pts, int64_t n, double rT, double rE)
{
    qsort(pts, (size_t)n, sizeof(or_pt), cmp_pt);
    double hv = 0.0, run = rE, pt = 0.0, pe = 0.0;
    int have = 0;
    for (int64_t i = 0; i < n; i++) {
        if (!(pts[i].t < rT) || !(pts[i].e < rE)) continue;
        if (pts[i].e < run) {
            if (have) hv = hv + (pts[i].t - pt) * (rE - pe);
            pt = pts[i].t;
            pe = pts[i].e;
            run = pe;
            have = 1;
        }
    }
    if (have) hv = hv + (rT - pt) * (rE - pe);
    return hv;
}

int oracle_hypervolume(int64_t n, const double *T, const double *E, double rT, double rE,
                       double *hv_out)
{
    if (n < 0) return OR_EINVAL;
    or_pt *p = (or_pt *)malloc(sizeof(or_pt) * (size_t)(n > 0 ? n : 1));
    if (!p) return OR_EINVAL;
    for (int64_t i = 0; i < n; i++) {
        p[i].t = T[i];
        p[i].e = E[i];
    }
    *hv_out = hv_of(p, n, rT, rE);
    free(p);
    return OR_OK;
}

/*
 * The three exploitation scores of Algorithm 1 for every unmeasured candidate of every
 * partition.  Energy variants (Sections 2.1 and 4.3): static energy is static power
 * times time, dynamic energy is total minus static:
 *     v = 0 total   E
 *     v = 1 dynamic E - p_static * T
 *     v = 2 static  p_static * T
 * Readings: for variant v, the current frontier is that of the measured points in the
 * (T, energy_v) plane, and the reference point is r_v = (1.1 * max T, 1.1 * max
 * energy_v) over the measured points (Appendix C).  Candidate y is (T_hat, energy_v of
 * (T_hat, E_hat)).
 *
 * Partition g owns candidates [cand_off[g], cand_off[g+1]) and measured points
 * [obs_off[g], obs_off[g+1]) (at least one).  Outputs: hvi[v * n_cand + x],
 * hv[g * 3 + v] = HV of the measured points, ref[g * 4 + 0] = rT and
 * ref[g * 4 + 1 + v] = rE_v.
 */
static double energy_variant(int v, double t, double e, double ps)
{
    if (v == 0) return e;
    if (v == 1) return e - ps * t;
    return ps * t;
}

int oracle_hvi(int n_seg, const int64_t *cand_off, const double *T_hat, const double *E_hat,
               const int64_t *obs_off, const double *T_obs, const double *E_obs,
               double p_static, double *hvi, double *hv, double *ref)
{
    if (n_seg < 0) return OR_EINVAL;
    int64_t n_cand = n_seg > 0 ? cand_off[n_seg] : 0;
    for (int g = 0; g < n_seg; g++)
        if (obs_off[g + 1] - obs_off[g] < 1 || cand_off[g + 1] < cand_off[g]) return OR_EINVAL;
    int64_t max_obs = 0;
    for (int g = 0; g < n_seg; g++)
        if (obs_off[g + 1] - obs_off[g] > max_obs) max_obs = obs_off[g + 1] - obs_off[g];
    or_pt *p = (or_pt *)malloc(sizeof(or_pt) * (size_t)(max_obs + 1));
    if (!p) return OR_EINVAL;
    for (int g = 0; g < n_seg; g++) {
        int64_t o0 = obs_off[g], no = obs_off[g + 1] - o0;
        double mt = T_obs[o0];
        for (int64_t i = 1; i < no; i++)
            if (T_obs[o0 + i] > mt) mt = T_obs[o0 + i];
        double rT = 1.1 * mt;
        ref[g * 4] = rT;
        for (int v = 0; v < 3; v++) {
            double me = energy_variant(v, T_obs[o0], E_obs[o0], p_static);
            for (int64_t i = 1; i < no; i++) {
                double ev = energy_variant(v, T_obs[o0 + i], E_obs[o0 + i], p_static);
                if (ev > me) me = ev;
            }
            double rE = 1.1 * me;
            ref[g * 4 + 1 + v] = rE;
            for (int64_t i = 0; i < no; i++) {
                p[i].t = T_obs[o0 + i];
                p[i].e = energy_variant(v, T_obs[o0 + i], E_obs[o0 + i], p_static);
            }
            double base = hv_of(p, no, rT, rE);
            hv[g * 3 + v] = base;
            for (int64_t x = cand_off[g]; x < cand_off[g + 1]; x++) {
                for (int64_t i = 0; i < no; i++) {
                    p[i].t = T_obs[o0 + i];
                    p[i].e = energy_variant(v, T_obs[o0 + i], E_obs[o0 + i], p_static);
                }
                p[no].t = T_hat[x];
                p[no].e = energy_variant(v, T_hat[x], E_hat[x], p_static);
                hvi[(int64_t)v * n_cand + x] = hv_of(p, no + 1, rT, rE) - base;
            }
        }
    }
    free(p);
    return OR_OK;
}

/*
 * Exploration score of Algorithm 1: the standard deviation of the M ensemble
 * predictions of time plus that of energy.  Reading: population standard deviation
 * (divide by M), mean and squared deviations summed in member order.
 * Tm, Em [M][n] (member-major); unc [n].
 */
int oracle_uncertainty(int M, int64_t n, const double *Tm, const double *Em, double *unc)
{
    if (M < 1 || n < 0) return OR_EINVAL;
    for (int64_t x = 0; x < n; x++) {
        double st = 0.0, se = 0.0;
        for (int m = 0; m < M; m++) {
            st = st + Tm[(int64_t)m * n + x];
            se = se + Em[(int64_t)m * n + x];
        }
        double mt = st / M, me = se / M;
        double vt = 0.0, ve = 0.0;
        for (int m = 0; m < M; m++) {
            double dt = Tm[(int64_t)m * n + x] - mt, de = Em[(int64_t)m * n + x] - me;
            vt = vt + dt * dt;
            ve = ve + de * de;
        }
        unc[x] = sqrt(vt / M) + sqrt(ve / M);
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------------
 * Multi-pass candidate selection of Algorithm 1, per partition:
 *     C = TopK(score_0 over X \ D, k1)
 *     C = C u TopK(score_1 over X \ D, k2)
 *     C = C u TopK(score_2 over X \ D, k3)
 *     C = C u TopK(unc over X \ D \ C, k - |C|)        (skipped when unc is NULL)
 * TopK(s over A, m) takes the m members of A with the largest s, ties to the smaller
 * index (all of A if it has fewer than m).  X is the partition's candidates (local
 * indices 0..n_g-1), D the measured ones: obs_idx[obs_off[g] .. obs_off[g+1]) hold
 * local indices; entries outside [0, n_g) name no candidate and are ignored.  C is
 * written in the order the passes add it (each pass by rank, members already in C
 * skipped) to sel[g * k ...], its size to count[g].  score [3][n_cand], unc [n_cand].
 * Needs 0 <= k1, k2, k3, k1 + k2 + k3 <= k; any NaN score is an error.
 * ---------------------------------------------------------------------------- */
static int cmp_score(const void *a, const void *b, void *ctx)
{
    const double *sc = (const double *)ctx;
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    if (sc[x] > sc[y]) return -1;
    if (sc[x] < sc[y]) return 1;
    return (x > y) - (x < y);
}

int oracle_select(int n_seg, const int64_t *cand_off, const double *score, const double *unc,
                  const int64_t *obs_off, const int64_t *obs_idx, int k1, int k2, int k3, int k,
                  int64_t *sel, int32_t *count)
{
    if (n_seg < 0 || k1 < 0 || k2 < 0 || k3 < 0 || k1 + k2 + k3 > k) return OR_EINVAL;
    int64_t n_cand = n_seg > 0 ? cand_off[n_seg] : 0;
    for (int64_t x = 0; x < n_cand; x++) {
        if (score[x] != score[x] || score[n_cand + x] != score[n_cand + x] ||
            score[2 * n_cand + x] != score[2 * n_cand + x])
            return OR_EINVAL;
        if (unc && unc[x] != unc[x]) return OR_EINVAL;
    }
    for (int g = 0; g < n_seg; g++) {
        int64_t c0 = cand_off[g], ng = cand_off[g + 1] - c0;
        char *in_d = (char *)calloc((size_t)(ng > 0 ? ng : 1), 1);
        char *in_c = (char *)calloc((size_t)(ng > 0 ? ng : 1), 1);
        int64_t *a = (int64_t *)malloc(sizeof(int64_t) * (size_t)(ng > 0 ? ng : 1));
        if (!in_d || !in_c || !a) {
            free(in_d);
            free(in_c);
            free(a);
            return OR_EINVAL;
        }
        for (int64_t i = obs_off[g]; i < obs_off[g + 1]; i++)
            if (obs_idx[i] >= 0 && obs_idx[i] < ng) in_d[obs_idx[i]] = 1;
        int32_t cnt = 0;
        int want[3] = {k1, k2, k3};
        for (int pass = 0; pass < 4; pass++) {
            if (pass == 3 && !unc) break;
            const double *s = pass < 3 ? score + (int64_t)pass * n_cand + c0 : unc + c0;
            int64_t na = 0;
            for (int64_t x = 0; x < ng; x++)
                if (!in_d[x] && !(pass == 3 && in_c[x])) a[na++] = x;
            qsort_r(a, (size_t)na, sizeof(int64_t), cmp_score, (void *)s);
            int64_t m = pass < 3 ? want[pass] : k - cnt;
            if (m > na) m = na;
            for (int64_t r = 0; r < m; r++) {
                if (in_c[a[r]]) continue;
                in_c[a[r]] = 1;
                sel[(int64_t)g * k + cnt++] = a[r];
            }
        }
        count[g] = cnt;
        free(in_d);
        free(in_c);
        free(a);
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------------
 * Stopping rule of Algorithm 1 (Appendix C): after batch b the relative HV improvement
 * is (hv[b] - hv[b-1]) / hv[b-1]; stop once the mean of the last R of them is below
 * eps.  hv[0] is the HV after the initial sample, hv[1..n-1] after each batch.
 * Reading: with hv[b-1] = 0 the relative improvement is +inf (never converged).
 * Returns 1 to stop after the last batch, 0 to go on.
 * ---------------------------------------------------------------------------- */
int oracle_hv_converged(int n, const double *hv, int R, double eps)
{
    if (R < 1 || n - 1 < R) return 0;
    double s = 0.0;
    for (int b = n - R; b < n; b++) {
        if (!(hv[b - 1] != 0.0)) return 0;
        s = s + (hv[b] - hv[b - 1]) / hv[b - 1];
    }
    return s / R < eps;
}

/* ------------------------------------------------------------------------------
 * Frontier comparison metrics of the evaluation (Section 6.1, "Metrics"): baseline
 * point set A against point set B, all in percent of the baseline's value.
 *   out[0], out[1]  max-throughput comparison: time and energy reduction of B's
 *                   leftmost point against A's (leftmost = least time, ties to the
 *                   least energy)
 *   out[2]          iso-time energy reduction: deadline d = A's least time;
 *                   E_X(d) = least energy among X's points with time <= d
 *   out[3]          iso-energy time reduction: budget b = A's least energy;
 *                   T_X(b) = least time among X's points with energy <= b
 *   out[4..6]       d, E_A(d), E_B(d);   out[7..9]  b, T_A(b), T_B(b)
 * A reduction is (base - x) / base * 100; NaN when B has no point within the deadline
 * or budget.  A and B need at least one point each.
 * ---------------------------------------------------------------------------- */
int oracle_compare(int64_t nA, const double *TA, const double *EA, int64_t nB,
                   const double *TB, const double *EB, double *out)
{
    if (nA < 1 || nB < 1) return OR_EINVAL;
    int64_t la = 0, lb = 0;
    for (int64_t i = 1; i < nA; i++)
        if (TA[i] < TA[la] || (TA[i] == TA[la] && EA[i] < EA[la])) la = i;
    for (int64_t i = 1; i < nB; i++)
        if (TB[i] < TB[lb] || (TB[i] == TB[lb] && EB[i] < EB[lb])) lb = i;
    out[0] = (TA[la] - TB[lb]) / TA[la] * 100.0;
    out[1] = (EA[la] - EB[lb]) / EA[la] * 100.0;
    double d = TA[la];
    double ea = INFINITY, eb = INFINITY;
    for (int64_t i = 0; i < nA; i++)
        if (TA[i] <= d && EA[i] < ea) ea = EA[i];
    for (int64_t i = 0; i < nB; i++)
        if (TB[i] <= d && EB[i] < eb) eb = EB[i];
    if (eb == INFINITY) eb = NAN;
    out[2] = (ea - eb) / ea * 100.0;
    out[4] = d;
    out[5] = ea;
    out[6] = eb;
    double b = EA[0];
    for (int64_t i = 1; i < nA; i++)
        if (EA[i] < b) b = EA[i];
    double ta = INFINITY, tb = INFINITY;
    for (int64_t i = 0; i < nA; i++)
        if (EA[i] <= b && TA[i] < ta) ta = TA[i];
    for (int64_t i = 0; i < nB; i++)
        if (EB[i] <= b && TB[i] < tb) tb = TB[i];
    if (tb == INFINITY) tb = NAN;
    out[3] = (ta - tb) / ta * 100.0;
    out[7] = b;
    out[8] = ta;
    out[9] = tb;
    return OR_OK;
}

/* ------------------------------------------------------------------------------
 * Launch-timing frontier of two operation sequences (Appendix B's dynamic program).
 *
 * S1 = ops[0 .. I-1] and S2 = ops[I .. I+J-1] run in their own order; ops of different
 * sequences are independent.  kind[o] = 0 for a computation, 1 for a communication (a
 * run of consecutive collectives counts as one).  Per op, ops[o*4 + 0..3]:
 *   computation: time and dynamic power alone (all SMs), time and dynamic power while
 *                a communication holds its SMs;
 *   communication: time and dynamic power (with its SM allocation), unused, unused.
 * A schedule is a sequence of groups, each one of
 *   case 0: the next op of S1 alone;  case 1: the next op of S2 alone;
 *   case 2: the next op of S1, a communication, overlapped with the next k (1 .. Kmax)
 *           ops of S2, all computations;
 *   case 3: the same with the roles of S1 and S2 swapped.
 * Groups run one after another; a schedule's time and energy are the sums over its
 * groups.  P(i, j), the frontier of the suffixes from S1[i] and S2[j], is GetFrontier of
 * (group cost + point of the successor cell) over every case, with P(I, J) = {(0, 0)}.
 *
 * Readings (the appendix leaves these open): overlap only pairs a communication with
 * computations; within an overlapped group both start together, the computations run
 * in order in the shared state until the communication ends and alone after it (the
 * fluid progress of the partition cost model), and the group ends when both are done;
 * every group's energy is its dynamic energy plus static power times its time.
 *
 * Floating-point order: group time/energy as written in group_cost; a candidate is
 * (g.T + p.T, g.E + p.E).  Candidates are generated by case (0, 1, 2 by k, 3 by k) and,
 * within one, by the successor's points in ascending time; GetFrontier keeps the first
 * of exact duplicates.  Output: P(0, 0) in ascending time with each point's schedule
 * as codes case * 32 + k (k = 0 for a lone op), padded with -1 to I + J entries;
 * stats[0] = the largest frontier of any cell, stats[1] = the frontier points of all
 * cells together, stats[2] = the most candidates of any cell.
 * ---------------------------------------------------------------------------- */
typedef struct { double T, E; int32_t src, q; } dp_pt;

typedef struct {
    int ncase, k, ni, nj;  /* decision and successor cell */
    double T, E;
} dp_src;

static void group_cost(const double *ops, int comm, const int *run, int k, double ps, double *T,
                       double *E)
{
    const double *c = ops + 4 * comm;
    double tc = c[0], pc = c[1];
    double tau = 0.0, e = 0.0;
    for (int r = 0; r < k; r++) {
        const double *o = ops + 4 * run[r];
        double t0 = o[0], p0 = o[1], t1 = o[2], p1 = o[3];
        if (tau < tc) {
            double nt = tau + t1;
            if (nt <= tc) {
                e = e + t1 * p1;
                tau = nt;
            } else {
                double dt = tc - tau;
                double rem = 1.0 - dt / t1;
                double ta = rem * t0;
                e = e + dt * p1;
                e = e + ta * p0;
                tau = tc + ta;
            }
        } else {
            e = e + t0 * p0;
            tau = tau + t0;
        }
    }
    double t = tau > tc ? tau : tc;
    *T = t;
    *E = (e + tc * pc) + ps * t;
}

static void alone_cost(const double *ops, int o, double ps, double *T, double *E)
{
    double t = ops[4 * o], p = ops[4 * o + 1];
    *T = t;
    *E = t * p + ps * t;
}

static int cmp_dp(const void *a, const void *b)
{
    const dp_pt *x = (const dp_pt *)a, *y = (const dp_pt *)b;
    if (x->T < y->T) return -1;
    if (x->T > y->T) return 1;
    if (x->E < y->E) return -1;
    if (x->E > y->E) return 1;
    /* candidate order: src then q (the order they were generated in) */
    if (x->src != y->src) return x->src < y->src ? -1 : 1;
    return (x->q > y->q) - (x->q < y->q);
}

int oracle_launch_dp(int I, int J, const int32_t *kind, const double *ops, double ps, int Kmax,
                     int64_t cap, double *oT, double *oE, int32_t *osched, int64_t *n_out,
                     int64_t *stats)
{
    if (I < 0 || J < 0 || I + J < 1 || Kmax < 0 || cap < 0) return OR_EINVAL;
    int W = J + 1;
    int ncell = (I + 1) * (J + 1);
    dp_pt **cell = (dp_pt **)calloc((size_t)ncell, sizeof(dp_pt *));
    int *cnt = (int *)calloc((size_t)ncell, sizeof(int));
    dp_src **srcs = (dp_src **)calloc((size_t)ncell, sizeof(dp_src *));
    int *run = (int *)malloc(sizeof(int) * (size_t)(I + J + 1));
    int rc = OR_OK;
    if (!cell || !cnt || !srcs || !run) { rc = OR_EINVAL; goto done; }
    stats[0] = 1;
    stats[1] = 1;
    stats[2] = 0;
    cell[I * W + J] = (dp_pt *)malloc(sizeof(dp_pt));
    cell[I * W + J][0].T = 0.0;
    cell[I * W + J][0].E = 0.0;
    cell[I * W + J][0].src = -1;
    cell[I * W + J][0].q = -1;
    cnt[I * W + J] = 1;
    for (int i = I; i >= 0; i--) {
        for (int j = J; j >= 0; j--) {
            if (i == I && j == J) continue;
            dp_src *s = (dp_src *)malloc(sizeof(dp_src) * (size_t)(2 + 2 * (Kmax + 1)));
            int ns = 0;
            if (i < I) {
                s[ns].ncase = 0; s[ns].k = 0; s[ns].ni = i + 1; s[ns].nj = j;
                alone_cost(ops, i, ps, &s[ns].T, &s[ns].E);
                ns++;
            }
            if (j < J) {
                s[ns].ncase = 1; s[ns].k = 0; s[ns].ni = i; s[ns].nj = j + 1;
                alone_cost(ops, I + j, ps, &s[ns].T, &s[ns].E);
                ns++;
            }
            if (i < I && kind[i] == 1) {
                for (int k = 1; k <= Kmax && j + k <= J; k++) {
                    if (kind[I + j + k - 1] != 0) break;
                    for (int r = 0; r < k; r++) run[r] = I + j + r;
                    s[ns].ncase = 2; s[ns].k = k; s[ns].ni = i + 1; s[ns].nj = j + k;
                    group_cost(ops, i, run, k, ps, &s[ns].T, &s[ns].E);
                    ns++;
                }
            }
            if (j < J && kind[I + j] == 1) {
                for (int k = 1; k <= Kmax && i + k <= I; k++) {
                    if (kind[i + k - 1] != 0) break;
                    for (int r = 0; r < k; r++) run[r] = i + r;
                    s[ns].ncase = 3; s[ns].k = k; s[ns].ni = i + k; s[ns].nj = j + 1;
                    group_cost(ops, I + j, run, k, ps, &s[ns].T, &s[ns].E);
                    ns++;
                }
            }
            int nc = 0;
            for (int a = 0; a < ns; a++) nc += cnt[s[a].ni * W + s[a].nj];
            dp_pt *cand = (dp_pt *)malloc(sizeof(dp_pt) * (size_t)(nc > 0 ? nc : 1));
            int w = 0;
            for (int a = 0; a < ns; a++) {
                const dp_pt *succ = cell[s[a].ni * W + s[a].nj];
                for (int q = 0; q < cnt[s[a].ni * W + s[a].nj]; q++) {
                    cand[w].T = s[a].T + succ[q].T;
                    cand[w].E = s[a].E + succ[q].E;
                    cand[w].src = a;
                    cand[w].q = q;
                    w++;
                }
            }
            qsort(cand, (size_t)nc, sizeof(dp_pt), cmp_dp);
            double best = INFINITY;
            int kept = 0;
            for (int c = 0; c < nc; c++)
                if (cand[c].E < best) {
                    best = cand[c].E;
                    cand[kept++] = cand[c];
                }
            cell[i * W + j] = cand;
            cnt[i * W + j] = kept;
            srcs[i * W + j] = s;
            if (kept > stats[0]) stats[0] = kept;
            stats[1] += kept;
            if (nc > stats[2]) stats[2] = nc;
        }
    }
    *n_out = cnt[0];
    for (int q = 0; q < cnt[0] && q < cap; q++) {
        oT[q] = cell[0][q].T;
        oE[q] = cell[0][q].E;
        int32_t *sc = osched + (int64_t)q * (I + J);
        for (int d = 0; d < I + J; d++) sc[d] = -1;
        int ci = 0, cj = 0, cq = q, d = 0;
        while (!(ci == I && cj == J)) {
            const dp_pt *p = &cell[ci * W + cj][cq];
            const dp_src *a = &srcs[ci * W + cj][p->src];
            sc[d++] = a->ncase * 32 + a->k;
            ci = a->ni;
            cj = a->nj;
            cq = p->q;
        }
    }
done:
    if (cell)
        for (int c = 0; c < ncell; c++) free(cell[c]);
    if (srcs)
        for (int c = 0; c < ncell; c++) free(srcs[c]);
    free(cell);
    free(cnt);
    free(srcs);
    free(run);
    return rc;
}
