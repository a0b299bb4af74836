/*
 * fs_oracle.h -- plain, slow CPU oracle for FleetSieve's allocation solve,
 * acquisition score and decision certificate.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library
 * and its Python binding) may include, link or call this code; only the
 * tests, the smoke check and the CPU-baseline leg of the benchmark do.
 * It shares no code with the GPU path.
 *
 * Precision: IEEE binary32 for every fulfillment value (the GPU path must
 * reproduce it bit for bit), binary64 for gaps and scores.  Build with
 * -ffp-contract=off and without fast-math.
 *
 * Cell layout, shared with the library's public contract:
 *   cell(i, t, b) = (i * n_tp + t) * n_levels + b
 * for class i, TP index t (into the ascending tp[] array) and load level b.
 */
#ifndef FS_ORACLE_H
#define FS_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORC_MAX_CLASSES 64
#define ORC_MAX_TP 8
#define ORC_MAX_LEVELS 32
#define ORC_MAX_BUDGET 4096

/* Problem statement (Section 3): classes with demand lambda_i and SLO L_i,
 * the TP set, the per-replica load grid and the GPU budget G. */
typedef struct orc_problem {
  int32_t n_classes, n_tp, n_levels, budget; /* K, |T|, B, G */
  const int32_t *tp;        /* [n_tp] GPUs per replica, ascending          */
  const float *levels;      /* [n_levels] per-replica load grid, ascending */
  const float *demand;      /* [K] lambda_i, req/s                         */
  const float *slo;         /* [K] L_i, tail limit                         */
  const float *floor_rps;   /* [K] critical floor in req/s (0 = none), or NULL */
} orc_problem;

/* One class's choice: TP index (-1 = empty), replicas (0 = empty). */
typedef struct orc_alloc {
  float tau;       /* max-min fulfillment, objective level (2)        */
  int32_t floors_met;
  int32_t gpus;    /* total GPUs used                                  */
  float goodput;   /* sum of served req/s in class order (fp32)        */
  int32_t tp_index[ORC_MAX_CLASSES];
  int32_t replicas[ORC_MAX_CLASSES];
} orc_alloc;

enum { ORC_UNDECIDED = 0, ORC_CERTIFIED_FEASIBLE = 1, ORC_CERTIFIED_INFEASIBLE = 2 };

/* Returns 0 when the problem is well formed, -1 otherwise. */
int orc_check_problem(const orc_problem *p);

/* Load bucket of replica count r for class i, or -1 when r replicas cannot
 * carry the class at any level of the grid. */
int orc_bucket(const orc_problem *p, int i, int r);

/* Fulfillment of one option on a point realisation. */
float orc_fulfillment(const orc_problem *p, int i, float cap, float tail, int r);

/* Three independent solvers of the same allocation problem on one point
 * realisation cap[N], tail[N].  All return 0 on success.
 *   brute:     enumerates every combination (tiny inputs only);
 *   dp:        (max,min) knapsack over the budget, then canonical allocation;
 *   threshold: largest achievable value whose minimum GPU need fits in G
 *              (returns tau only; the allocation fields are left zero). */
int orc_solve_brute(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out);
int orc_solve_dp(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out);
int orc_solve_threshold(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out);

/* Dense batch: scenario j is cap[j*N..], tail[j*N..].  Uses orc_solve_dp. */
int orc_solve_batch(const orc_problem *p, const float *cap, const float *tail, int64_t n,
                    orc_alloc *out, int n_threads);

/* Acquisition score (Section 4.3) for n_orders reveal orders.
 * Intervals and measured flags are [O][N]; cand is [E] cell indices;
 * samples are [O][E][S].  Outputs: score[O][E], gap_now[O], best[O],
 * tau_dump [O][E][S][2] (tau-, tau+) or NULL.
 * Only tiles (o, e) with tile_mask[o*E+e] != 0 are solved when tile_mask is
 * not NULL; the others are left untouched in score and tau_dump. */
int orc_score(const orc_problem *p, int32_t n_orders,
              const float *cap_lo, const float *cap_hi,
              const float *tail_lo, const float *tail_hi, const uint8_t *measured,
              const int32_t *cand, int32_t n_cand,
              const float *cap_s, const float *tail_s, int32_t n_samples,
              double *score, double *gap_now, int32_t *best, float *tau_dump,
              const uint8_t *tile_mask, int n_threads);

/* Three-state certificate (Section 4.2) per order. */
int orc_certify(const orc_problem *p, int32_t n_orders,
                const float *cap_lo, const float *cap_hi,
                const float *tail_lo, const float *tail_hi, const uint8_t *measured,
                float eps, int32_t *state, orc_alloc *cons, orc_alloc *opt, double *gap);

/* The paper's whole lexicographic objective (Section 3): levels (1) floors
 * and (2) max-min fulfillment as above, then (3) the largest total served
 * goodput among allocations that keep every class's ratio at least tau*
 * (and the floors), then (4) the fewest GPUs; remaining ties go to the
 * lexicographically smallest (t_0, r_0, t_1, r_1, ...) in class order with
 * t the TP degree and empty = (0, 0).  A class's served goodput is
 * min(lambda, fl32(r c)) when its tail is within the SLO, else 0; the total
 * compared at level (3) is their binary64 sum accumulated from the last
 * class to the first, returned in *goodput64 (may be NULL).
 *   lex_brute: every combination, keys compared literally (tiny inputs);
 *   lex:       levels (1)-(2) by orc_solve_dp, then a suffix knapsack over
 *              the budget and a greedy reconstruction in class order. */
int orc_solve_lex_brute(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out,
                        double *goodput64);
int orc_solve_lex(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out,
                  double *goodput64);

/* Certificate with the stage-wise gap (Section 4.2): both allocations under
 * the whole objective; gap_mm = tau+ - tau-, gap_gp = |gp+ - gp-| /
 * max(gp+, gp-) (0 when both are 0) in binary64; CERTIFIED_FEASIBLE needs
 * both stages within eps. */
int orc_certify_lex(const orc_problem *p, int32_t n_orders, const float *cap_lo, const float *cap_hi,
                    const float *tail_lo, const float *tail_hi, const uint8_t *measured, float eps,
                    int32_t *state, orc_alloc *cons, orc_alloc *opt, double *gap_mm, double *gap_gp);

/* Acquisition score with the stage-wise gap (Section 4.3 with Section 4.2's
 * stages) under the whole objective: per (order, candidate) the expected
 * reduction of each stage, score_mm = gap_mm - mean Gamma_mm(s) and score_gp
 * = gap_gp - mean Gamma_gp(s) (pairwise sums over the samples), gap_* the
 * order's current stages; best = the larger score_mm, then the larger
 * score_gp, then the smaller TP, cell index, candidate.  Measured candidates
 * score (0, 0) and are never picked. */
int orc_score_lex(const orc_problem *p, int32_t n_orders, const float *cap_lo, const float *cap_hi,
                  const float *tail_lo, const float *tail_hi, const uint8_t *measured, const int32_t *cand,
                  int32_t n_cand, const float *cap_s, const float *tail_s, int32_t n_samples, double *score_mm,
                  double *score_gp, double *gap_mm, double *gap_gp, int32_t *best, const uint8_t *tile_mask,
                  int n_threads);

/* Pairwise sum of x[0..n) zero-padded to the next power of two. */
double orc_pairwise_sum(const double *x, int64_t n);

#ifdef __cplusplus
}
#endif
#endif
