/*
 * fleetsieve.h -- C ABI of libfleetsieve, an MI355X (gfx950) implementation
 * of FleetSieve's decision-critical acquisition scorer.
 *
 * The method (Sections 3-4 of the FleetSieve paper): a fleet planner assigns
 * each workload class i one serving configuration -- a TP degree t and a
 * replica count r -- under a GPU budget G, maximising the minimum satisfaction
 * ratio over classes.  Performance of a (class, TP, load) cell is uncertain:
 * capacity lies in [c_lo, c_hi] and the tail metric in [l_lo, l_hi].  The
 * planner solves a conservative realisation (c_lo, l_hi) and an optimistic one
 * (c_hi, l_lo); the gap between their objectives is what profiling must close.
 * Each unmeasured cell is scored by the expected gap reduction its
 * measurement would bring, estimated over sampled outcomes.
 *
 * Conventions for every call:
 *   - Array arguments are DEVICE pointers owned by the caller, except the
 *     fs_problem struct and what it points to, which are HOST memory read
 *     during the call only.
 *   - Work is enqueued on the caller's stream; the call returns without
 *     synchronising.  Outputs are valid once the stream reaches that point.
 *     The library allocates no device memory per call: temporary state lives
 *     in a caller-provided workspace of at least fs_workspace_size() bytes,
 *     which must not be used by anything else until the stream has passed
 *     the call.
 *   - The returned status covers argument validation and launch errors.  On
 *     any status other than FS_OK nothing was enqueued and fs_last_error()
 *     (thread-local) describes the problem.  No exception crosses the ABI.
 *   - Numerics: every fulfillment value is the IEEE binary32 result of one
 *     multiply and one correctly rounded divide, bit-identical to a plain
 *     binary32 CPU evaluation; gaps and scores are binary64 with a fixed
 *     summation order.  Results are deterministic run to run.
 *
 * Cell layout: cell(i, t, b) = (i * n_tp + t) * n_levels + b for class i,
 * TP index t (into the ascending tp[] array) and load level b; N cells.
 */
#ifndef FLEETSIEVE_H
#define FLEETSIEVE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FS_MAX_CLASSES 64
#define FS_MAX_TP 8
#define FS_MAX_LEVELS 32
#define FS_MAX_BUDGET 4096
#define FS_MAX_SAMPLES (1 << 20)
#define FS_TP_NONE 0xFF

typedef enum fs_status {
  FS_OK = 0,
  FS_ERR_INVALID_ARGUMENT = 1,
  FS_ERR_UNSUPPORTED = 2,
  FS_ERR_WORKSPACE_TOO_SMALL = 3,
  FS_ERR_DEVICE = 4,
  FS_ERR_INTERNAL = 5
} fs_status;

/* The three states of the decision certificate (Section 4.2). */
typedef enum fs_cert {
  FS_UNDECIDED = 0,
  FS_CERTIFIED_FEASIBLE = 1,
  FS_CERTIFIED_INFEASIBLE = 2
} fs_cert;

/* The allocation problem of Section 3 (host memory).
 * Requirements (FS_ERR_INVALID_ARGUMENT otherwise):
 *   1 <= n_classes <= 64, 1 <= n_tp <= 8, 1 <= n_levels <= 32,
 *   tp[0] <= budget <= 4096; tp strictly ascending and >= 1; levels strictly
 *   ascending, finite, > 0; demand in [2^-32, 2^32]; slo not NaN (+inf
 *   allowed); floor_rps NULL or finite and >= 0 (0 = not a critical class).
 * Device-side cell values must be finite and >= 0 with capacities 0 or in
 * [2^-64, 2^64] (tails may be +inf); this keeps every quotient a normal
 * binary32 number.  They are checked only when the environment variable
 * FS_VALIDATE=1 is set, which adds a synchronous check per call. */
typedef struct fs_problem {
  int32_t n_classes;       /* K: workload classes                                */
  int32_t n_tp;            /* |T|: candidate TP degrees                          */
  int32_t n_levels;        /* B: per-replica load levels                         */
  int32_t budget;          /* G: GPUs in the fleet (Eq. 3)                       */
  const int32_t *tp;       /* [n_tp] GPUs per replica                            */
  const float *levels;     /* [n_levels] per-replica load grid, req/s            */
  const float *demand;     /* [K] lambda_i, offered demand, req/s                */
  const float *slo;        /* [K] L_i, limit on the cell's tail metric (Eq. 5)   */
  const float *floor_rps;  /* [K] critical floor in served req/s, or NULL        */
} fs_problem;

/* Per-order uncertainty state (Section 4.1), device memory, each [n_orders][N].
 * A measured cell (measured = 1) has a point interval. */
typedef struct fs_intervals {
  const float *cap_lo, *cap_hi;    /* capacity bounds, req/s per replica     */
  const float *tail_lo, *tail_hi;  /* tail-metric bounds                     */
  const uint8_t *measured;         /* 1 = revealed                           */
} fs_intervals;

/* Allocation outputs, device memory, structure of arrays over n entries.
 * Any pointer may be NULL to skip that output. */
typedef struct fs_alloc {
  float *objective;     /* [n] max-min fulfillment tau*                          */
  uint8_t *tp_index;    /* [n][K] index into tp[], FS_TP_NONE = class unserved   */
  uint16_t *replicas;   /* [n][K] replica count, 0 = class unserved              */
  uint8_t *floors_met;  /* [n] 1 when every critical floor is met (or none exist)*/
  float *goodput;       /* [n] total served req/s, binary32 sum in class order   */
} fs_alloc;

typedef struct fs_context fs_context;

/* Options for fs_context_set_option. */
typedef enum fs_option {
  /* Scoring kernel: 0 = automatic (3 without critical floors, else 1),
   * 1 = one wavefront per scenario, full solves (any problem),
   * 2 = one lane per scenario, full solves (no floors, TP set {1,2,4,8},
   *     budget 16, 32 or 64),
   * 3 = exclusion scorer: per-order all-but-one tables, O(replica range) per
   *     scenario (no floors).  All give identical bits. */
  FS_OPT_SCORE_KERNEL = 1,
  /* n in [1, 64]: in every scoring call, launch the scoring kernel (the
   * per-scenario solves) n times back to back between a pair of HIP events
   * on the caller's stream, for fs_context_kernel_timing.  The kernel is
   * idempotent, so the outputs are those of one launch.  0 = off (default). */
  FS_OPT_KERNEL_TIMING = 2,
  /* Exclusion scorer (kernel 3): samples each lane handles, 4, 8 or 16
   * (0 = library default).  A launch-shape tuning knob; results are
   * identical for every value. */
  FS_OPT_SAMPLES_PER_LANE = 3,
  /* Exclusion scorer: wavefronts of its fixed grid, which stride over the
   * work items, in [1, 2^20] (0 = library default).  A launch-shape tuning
   * knob; results are identical for every value. */
  FS_OPT_SCORER_WAVES = 5,
  /* Exclusion scorer set-up: 0 = automatic (one block per order and
   * realisation when the budget is at most 64 GPUs, there are at most 16
   * classes and its LDS fits), 1 = the general set-up (one block per order,
   * realisation and class; any problem).  Results are identical. */
  FS_OPT_SETUP = 6,
  /* Objective of fs_profile_loop: FS_OBJECTIVE_MAXMIN (default; objective
   * levels 1-2, the max-min gap and score, as fs_certify and
   * fs_score_candidates) or FS_OBJECTIVE_LEXICOGRAPHIC (the whole objective:
   * the stage-wise certificate of fs_certify_lex and the stage-wise score of
   * fs_score_candidates_lex, which solves every scenario in full;
   * FS_ERR_UNSUPPORTED where that does not fit). */
  FS_OPT_LOOP_OBJECTIVE = 7,
  /* 1: fs_profile_loop starts every round with Algorithm 1's fit step,
   * fs_refit_intervals of each trajectory's initial intervals with its
   * revealed cells; the certificate and the score use the refitted
   * intervals and the samples clamped into them.  Needs the workspace of
   * fs_loop_refit_workspace_size.  0 (default): no refit. */
  FS_OPT_LOOP_REFIT = 8,
  /* Exclusion scorer set-up: where the search for each option's capacity
   * threshold (the smallest binary32 capacity at which the option reaches a
   * given ratio) starts: 0 (default) = a window of eight bit patterns around
   * the quotient estimate, then stepping, then a bisection over all bit
   * patterns; 1 = stepping, then bisection; 2 = bisection only.  Every value
   * gives identical results (a test knob for the later stages, which the
   * window leaves unused on ordinary inputs). */
  FS_OPT_THRESHOLD_SEARCH = 9
} fs_option;

typedef enum fs_objective { FS_OBJECTIVE_MAXMIN = 0, FS_OBJECTIVE_LEXICOGRAPHIC = 1 } fs_objective;

/* Creates a context bound to HIP device `hip_device` (with a stream and two
 * events of its own, used inside fs_score_candidates_lex).  One context per
 * host thread; a context is not thread-safe. */
fs_status fs_context_create(int hip_device, fs_context **out);
void fs_context_destroy(fs_context *ctx);
fs_status fs_context_set_option(fs_context *ctx, fs_option option, int64_t value);

/* Waits for the events recorded under FS_OPT_KERNEL_TIMING, returns the
 * summed time between each event pair in milliseconds and the number of
 * scoring-kernel launches they enclose, and forgets them. */
fs_status fs_context_kernel_timing(fs_context *ctx, double *total_ms, int64_t *launches);

/* Thread-local description of the last failure in this thread. */
const char *fs_last_error(void);

/* Host-only check of a problem statement (no device work). */
fs_status fs_validate_problem(const fs_problem *p);

/* Workspace bytes sufficient for any call on problem p with up to n_orders
 * orders, n_cand candidates and n_samples samples (pass 0 for unused). */
fs_status fs_workspace_size(const fs_problem *p, int32_t n_orders, int32_t n_cand,
                            int32_t n_samples, size_t *bytes);

/* Solves the allocation (Section 3, Eq. 1-5, objective levels (1)-(2) with
 * ties broken by fewer GPUs, then the lexicographically smaller TP vector) on
 * n_scenarios dense point realisations: scenario j uses cap[j*N .. j*N+N-1]
 * and tail[j*N ..].  Writes out.* for every scenario. */
fs_status fs_solve_batch(fs_context *ctx, const fs_problem *p, const float *d_cap,
                         const float *d_tail, int64_t n_scenarios, fs_alloc out,
                         void *d_workspace, size_t workspace_bytes, hipStream_t stream);

/* Acquisition scores (Section 4.3).  For order o, Gamma_t(o) is the gap
 * tau(optimistic) - tau(conservative) on the order's intervals.  Scenario
 * (o, e, s) replaces cell cand[e] in BOTH realisations by the sampled outcome
 * (cap_s, tail_s)[o][e][s]; its gap is Gamma(o, e, s).
 *   score[o][e] = Gamma_t(o) - (sum over s of Gamma(o, e, s)) / S
 * with the sum taken as a pairwise tree over s zero-padded to a power of two.
 * A candidate whose cell is measured in order o is not solved and scores
 * exactly 0.  best[o] is the unmeasured candidate with the largest score,
 * ties to the smaller profiling cost (TP degree of the cell), then the
 * smaller cell index, then the smaller e; -1 if none.
 *   d_cand    [n_cand] cell indices in [0, N)
 *   d_cap_s, d_tail_s  [n_orders][n_cand][n_samples]
 *   d_score   [n_orders][n_cand] binary64
 *   d_gap_now [n_orders] binary64 (may be NULL)
 *   d_best    [n_orders] int32 (may be NULL)
 *   d_tau_dump NULL or [n_orders][n_cand][n_samples][2] = (tau-, tau+); for a
 *             measured candidate it holds the order's base values.
 * Samples whose values cannot change the result are not read: the exclusion
 * scorer (kernel 3, the default without critical floors) skips a tile whose
 * cell no replica count reaches, and a tile whose tau is U in both
 * realisations whatever its samples (in the exclusion form of Section 3's
 * max-min knapsack: M at the range's first replica count at most U), and
 * forms their sums in closed form.
 * Limits: n_orders and n_cand in [0, 65535], n_samples in [1, 2^20]; the
 * exclusion scorer also needs n_orders * n_cand < 2^31 and returns
 * FS_ERR_UNSUPPORTED otherwise. */
fs_status fs_score_candidates(fs_context *ctx, const fs_problem *p, fs_intervals iv,
                              int32_t n_orders, const int32_t *d_cand, int32_t n_cand,
                              const float *d_cap_s, const float *d_tail_s, int32_t n_samples,
                              double *d_score, double *d_gap_now, int32_t *d_best,
                              float *d_tau_dump, void *d_workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* fs_score_candidates for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments and results without the workspace, which
 * is replaced by a static device array of FS_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs on until the process ends.  Sizes whose
 * fs_workspace_size exceeds it return FS_ERR_UNSUPPORTED.  Every call on one
 * GPU uses the same array: calls that overlap on one GPU (other streams, other
 * host threads) race and must be serialised by the caller.  The call makes
 * no allocation; it ignores FS_OPT_KERNEL_TIMING and the FS_VALIDATE check. */
#define FS_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
fs_status fs_score_candidates_noalloc(fs_context *ctx, const fs_problem *p, fs_intervals iv,
                                      int32_t n_orders, const int32_t *d_cand, int32_t n_cand,
                                      const float *d_cap_s, const float *d_tail_s, int32_t n_samples,
                                      double *d_score, double *d_gap_now, int32_t *d_best,
                                      float *d_tau_dump, hipStream_t stream);

/* Three-state certificate (Section 4.2, Algorithm 1) per order:
 *   CERTIFIED_INFEASIBLE if some class is critical and even the optimistic
 *     allocation cannot meet every critical floor;
 *   CERTIFIED_FEASIBLE if the conservative allocation meets the floors, every
 *     cell it commits to is measured with tail upper bound within the SLO,
 *     and the gap is at most eps;
 *   UNDECIDED otherwise.
 * Writes state [n_orders], the conservative (cons) and optimistic (opt)
 * allocations [n_orders] and the gap [n_orders] (binary64, may be NULL). */
fs_status fs_certify(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                     float eps, int32_t *d_state, fs_alloc cons, fs_alloc opt, double *d_gap,
                     void *d_workspace, size_t workspace_bytes, hipStream_t stream);

/* The paper's whole lexicographic objective (Section 3, after Eq. 5):
 * (1) critical floors whenever they can be met, (2) max-min fulfillment,
 * (3) the largest total served goodput among allocations that keep every
 * class's ratio at least tau* (and the floors), (4) the fewest GPUs; the
 * remaining ties go to the smallest (TP degree, replicas) of each class in
 * class order, an unserved class first.  A class's served goodput is
 * min(lambda, fl32(r c)) when the cell's tail is within the SLO, else 0;
 * level (3) compares their binary64 sum taken from the last class to the
 * first (exact while the nonzero served rates lie within a factor 2^23 of
 * each other).  fs_solve_batch and fs_certify use levels (1)-(2) with the
 * tie-breaks fewer GPUs, then smaller TP degrees.
 *
 * Supported while the solve's LDS fits 64 KiB: about (28 + 2K)(G + 1) +
 * 1 KiB (K = 4 up to G = 1787, K = 16 up to G = 1072, K = 64 up to G = 411);
 * FS_ERR_UNSUPPORTED otherwise.
 *
 * Dense batch under the whole objective: out as in fs_solve_batch (objective
 * = tau*, goodput = the binary32 class-order sum of the chosen allocation);
 * d_goodput64 [n] (or NULL) receives level (3)'s binary64 total. */
fs_status fs_solve_batch_lex(fs_context *ctx, const fs_problem *p, const float *d_cap, const float *d_tail,
                             int64_t n_scenarios, fs_alloc out, double *d_goodput64, void *d_workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* Certificate with the stage-wise allocation gap (Section 4.2; Fig. 4a
 * tracks both stages): A- and A+ under the whole objective; the max-min
 * stage tau+ - tau- and the goodput stage |gp+ - gp-| / max(gp+, gp-) (0
 * when both are 0), binary64, each [n_orders] or NULL.  CERTIFIED_FEASIBLE
 * needs both stages within eps; the other conditions are fs_certify's. */
fs_status fs_certify_lex(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders, float eps,
                         int32_t *d_state, fs_alloc cons, fs_alloc opt, double *d_gap_maxmin,
                         double *d_gap_goodput, void *d_workspace, size_t workspace_bytes, hipStream_t stream);

/* Acquisition score with the stage-wise gap under the whole objective
 * (Section 4.3's score over Section 4.2's stages): per scenario (order o,
 * candidate e, sample s) both allocations under the whole objective, the
 * max-min stage Gamma_mm = tau+ - tau- and the goodput stage Gamma_gp =
 * |gp+ - gp-| / max(gp+, gp-); per (o, e) the expected reduction of each,
 *   d_score_maxmin[o][e]  = gap_maxmin[o]  - (pairwise sum over s of Gamma_mm) / S,
 *   d_score_goodput[o][e] = gap_goodput[o] - (pairwise sum over s of Gamma_gp) / S;
 * d_best[o] = the largest max-min score, then the largest goodput score,
 * then the smaller TP, cell index, candidate (measured candidates score
 * (0, 0) and are never picked; -1 when none is left).  d_gap_*[o] (or NULL)
 * receive the order's current stages.  The max-min score equals
 * fs_score_candidates' score bit for bit.  By default the goodput stage of a
 * scenario comes from per-order tables (the best goodput of the other
 * classes per budget for every interval of the option ratios, built once per
 * call) plus the candidate cell's options at the sample; with
 * FS_OPT_SCORE_KERNEL set to 1, or where those tables do not fit, every scenario
 * is solved in full (two max-min solves and two knapsacks, one wavefront:
 * far slower).  Both give the same bits.  The orders' own stages are solved
 * on a second stream of the context, forked from and joined back into
 * `stream` within the call, so every output is ordered before later work on
 * `stream`.  Workspace: fs_score_lex_workspace_size; sizes as in
 * fs_score_candidates; FS_ERR_UNSUPPORTED where the whole objective does not
 * fit (see fs_solve_batch_lex). */
fs_status fs_score_lex_workspace_size(const fs_problem *p, int32_t n_orders, int32_t n_cand, int32_t n_samples,
                                      size_t *bytes);
fs_status fs_score_candidates_lex(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                                  const int32_t *d_cand, int32_t n_cand, const float *d_cap_s, const float *d_tail_s,
                                  int32_t n_samples, double *d_score_maxmin, double *d_score_goodput,
                                  double *d_gap_maxmin, double *d_gap_goodput, int32_t *d_best, void *d_workspace,
                                  size_t workspace_bytes, hipStream_t stream);

#define FS_MAX_METRICS 8

/* Class policy with several tail metrics and a success floor (Section 3,
 * Eq. 5 in full: a selected configuration must keep every tail metric within
 * its limit and its success probability at least s_min; Section 5 gives chat
 * success >= 99%, TTFT-p99 <= 2 s, completion-p99 <= 30 s).  Host memory. */
typedef struct fs_slo_policy {
  int32_t n_metrics;         /* M in [1, FS_MAX_METRICS]: tail metrics per cell        */
  const float *limit;        /* [K][M] limit of metric m for class i; +inf = none; not NaN */
  const float *success_min;  /* [K] success floor, or NULL (no success requirement)      */
} fs_slo_policy;

/* Feasibility of cells under a policy, as the single tail value every other
 * call tests: d_out[j][c] = 0 when every tail metric of cell c is within its
 * class's limit and (when floors are given) its success is at least the
 * floor, +inf otherwise (a NaN metric fails).  Given the problem with every
 * slo[i] = 0, the other calls then apply the policy exactly (0 <= 0 holds,
 * +inf <= 0 does not).  For intervals, reduce the conservative side (upper
 * tail bounds with the lower success bound) into tail_hi and the optimistic
 * side (lower tail bounds with the upper success bound) into tail_lo.
 *   d_tails   [n_rows][N][M] (metric fastest)
 *   d_success [n_rows][N] or NULL
 *   d_out     [n_rows][N] */
fs_status fs_reduce_cells(fs_context *ctx, const fs_problem *p, const fs_slo_policy *pol, const float *d_tails,
                          const float *d_success, int64_t n_rows, float *d_out, hipStream_t stream);

/* The same for candidate samples, each judged by its candidate's class:
 *   d_tail_s [n_orders][n_cand][n_samples][M], d_succ_s [n_orders][n_cand][n_samples] or NULL,
 *   d_out    [n_orders][n_cand][n_samples] (+inf for a candidate outside [0, N)).
 * n_orders and n_cand at most 65535, n_samples at most FS_MAX_SAMPLES.  With
 * n_samples a multiple of 4 and 16-byte aligned arrays the kernel moves 4
 * samples per 16-byte access. */
fs_status fs_reduce_samples(fs_context *ctx, const fs_problem *p, const fs_slo_policy *pol, const int32_t *d_cand,
                            int32_t n_cand, const float *d_tail_s, const float *d_succ_s, int32_t n_orders,
                            int32_t n_samples, float *d_out, hipStream_t stream);

/* Interval refit, Algorithm 1's fit step (Section 4.1: the intervals combine
 * an interior-knee structural prior with the measured cells).  The prior, as
 * read here: for every class and load level the capacity per GPU (c / t) is
 * unimodal over the TP degrees in ascending order, and for every class and
 * TP degree the tail does not fall as the load level rises.  For every
 * unmeasured cell (measured = point intervals, never written):
 *   cap_lo' = max(cap_lo, t * min(best measured c / t below t, best measured
 *             c / t above t)), binary64 rounded down to binary32, when
 *             measured TP degrees exist on both sides at the same class and
 *             level;
 *   tail_lo' = max(tail_lo, measured tails at lower levels, same class and TP),
 *   tail_hi' = min(tail_hi, measured tails at higher levels);
 * a bound that would empty the interval is dropped (the prior does not hold
 * there) and that quantity keeps its interval.  cap_hi and measured are
 * unchanged.  Outputs [n_orders][N] device arrays; each may alias its input
 * (cap_lo_out = iv.cap_lo etc. refits in place). */
fs_status fs_refit_intervals(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                             float *d_cap_lo_out, float *d_tail_lo_out, float *d_tail_hi_out, hipStream_t stream);

/* The candidates' samples moved into the candidates' current intervals
 * (Algorithm 1 refits the intervals every round; samples drawn once inside
 * the initial intervals are clamped into the refitted ones before scoring):
 *   cap_out[o][e][s]  = min(max(cap_s[o][e][s], cap_lo[o][c]), cap_hi[o][c]),
 *   tail_out[o][e][s] = min(max(tail_s[o][e][s], tail_lo[o][c]), tail_hi[o][c]),
 * with c = cand[e].  Arrays as in fs_score_candidates; each output
 * [n_orders][n_cand][n_samples] may alias its input.  The samples of a
 * candidate outside [0, N) are not written.  n_orders and n_cand in
 * [0, 65535], n_samples in [0, 2^20]. */
fs_status fs_clamp_samples(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                           const int32_t *d_cand, int32_t n_cand, const float *d_cap_s, const float *d_tail_s,
                           int32_t n_samples, float *d_cap_out, float *d_tail_out, hipStream_t stream);

/* Reveal rule of fs_profile_loop. */
typedef enum fs_policy {
  FS_POLICY_SCORE = 0,  /* the candidate with the largest score (Section 4.3, Algorithm 1) */
  FS_POLICY_ORDER = 1   /* the first unmeasured candidate of a caller-given order
                         * (for comparisons, e.g. a uniform random permutation) */
} fs_policy;

/* Duration of one profiling cell in seconds: a reveal costs this times the
 * cell's TP degree in GPU-seconds (Section 5). */
#define FS_CELL_SECONDS 300.0

/* Outputs of fs_profile_loop, device memory, one entry per trajectory. */
typedef struct fs_loop_out {
  int32_t *state;       /* [O] certificate state when the trajectory ended (fs_cert)       */
  uint8_t *finished;    /* [O] 1 = certified, or no unmeasured candidate was left;
                         *     0 = stopped by the round limit                               */
  int32_t *rounds;      /* [O] reveals made                                                 */
  double *gpu_seconds;  /* [O] FS_CELL_SECONDS x TP degree summed over the reveals          */
  int32_t *reveals;     /* [O][max_rounds] candidate revealed in each round, -1 after the
                         * end; or NULL                                                     */
  fs_alloc final_alloc; /* [O] the returned allocation (any field may be NULL): A- of the
                         * last certificate when the trajectory certified; otherwise
                         * Algorithm 1's best measured feasible allocation, the optimum
                         * of the table with every unmeasured cell infeasible            */
  float *tau_truth;     /* [O] objective level (2) of the returned allocation on the true
                         * table (smallest fulfillment over the classes, an unserved class
                         * counting 0); or NULL                                             */
  float *tau_oracle;    /* [O] optimum of the true table (fs_solve_batch); or NULL           */
} fs_loop_out;

/* Workspace bytes for fs_profile_loop with these sizes. */
/* Workspace of fs_profile_loop with FS_OPT_LOOP_REFIT = 1 (the loop's plus
 * the refitted intervals and two clamped copies of the samples). */
fs_status fs_loop_refit_workspace_size(const fs_problem *p, int32_t n_orders, int32_t n_cand, int32_t n_samples,
                                       size_t *bytes);

fs_status fs_loop_workspace_size(const fs_problem *p, int32_t n_orders, int32_t n_cand,
                                 int32_t n_samples, size_t *bytes);

/* The profiling loop (Algorithm 1) for n_orders independent trajectories.
 * Trajectory o starts from row o of iv (its initial design; iv is read only,
 * the loop works on a copy in the workspace).  Each round, for every
 * trajectory still running:
 *   1. the certificate (as fs_certify, tolerance eps);  a certified state
 *      (feasible or infeasible) ends the trajectory and returns A-;
 *   2. if no candidate is left unmeasured, the trajectory ends undecided and
 *      returns the best measured feasible allocation: the solve (under the
 *      loop's objective) of its table with every unmeasured cell infeasible
 *      and every measured cell at its measured values;
 *   3. otherwise one candidate is revealed: under FS_POLICY_SCORE the argmax
 *      of fs_score_candidates on the current intervals (same tie rule),
 *      under FS_POLICY_ORDER the first unmeasured candidate of
 *      d_order[o][0..n_cand) (entries outside [0, n_cand) are skipped).  Its
 *      cell's capacity and tail intervals collapse to the true values
 *      d_truth_cap[o][cell], d_truth_tail[o][cell] ([n_orders][N]), the cell
 *      becomes measured, and the trajectory is charged FS_CELL_SECONDS x TP.
 * After max_rounds reveals a trajectory gets one more certificate (steps 1-2)
 * and then stops (finished = 0 if still undecided, returning the best
 * measured feasible allocation as in step 2).  The intervals are not
 * refitted between rounds: the samples d_cap_s, d_tail_s
 * ([n_orders][n_cand][n_samples], drawn inside the initial intervals) stay
 * valid, since a candidate's intervals change only when it is revealed.
 * check_every > 0: every check_every rounds the call waits for the stream
 * and returns early once no trajectory is running (the call then returns
 * with the stream idle); check_every = 0: exactly max_rounds rounds are
 * enqueued without waiting.  Limits as fs_score_candidates; max_rounds in
 * [0, 65535]; critical floors are supported (the scorer then solves every
 * scenario in full). */
fs_status fs_profile_loop(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                          const float *d_truth_cap, const float *d_truth_tail,
                          const int32_t *d_cand, int32_t n_cand, const float *d_cap_s,
                          const float *d_tail_s, int32_t n_samples, float eps, fs_policy policy,
                          const int32_t *d_order, int32_t max_rounds, int32_t check_every,
                          fs_loop_out out, void *d_workspace, size_t workspace_bytes,
                          hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* FLEETSIEVE_H */
