// fs_internal.h -- structures shared by the host runtime and the gfx950
// kernels of libfleetsieve.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fs {

constexpr int kMaxClasses = 64;
constexpr int kMaxTp = 8;
constexpr int kMaxLevels = 32;
constexpr int kMaxBudget = 4096;
constexpr int kWave = 64;

// Problem constants, passed by value as a kernel argument (about 1.5 KB).
struct DevProblem {
  int32_t K, NT, B, G;
  int32_t N;          // cells = K * NT * B
  int32_t has_floor;  // some class has floor_rps > 0
  int32_t tp[kMaxTp];
  float levels[kMaxLevels];
  float demand[kMaxClasses];
  float slo[kMaxClasses];
  float floor_rps[kMaxClasses];
  // binary64 reciprocal of each demand, correctly rounded.  For binary32 x,
  // fl32(fl64(x * rcp)) equals the correctly rounded binary32 x / demand
  // whenever the quotient is a normal number (the binary64 error, at most
  // 2^-52 relative, is below the distance from any binary32 rounding
  // midpoint, at least 2^-50 relative).
  double rcp_demand[kMaxClasses];
  // First option of each TP degree among one class's options, which are
  // ordered by TP, then replicas: optoff[t] = sum over t' < t of G / tp[t'];
  // optoff[NT] is the number of options per class.
  int32_t optoff[kMaxTp + 1];
};

// Where a candidate cell enters the allocation: its class, TP index, load
// level, and the replica counts [rlo, rhi] whose per-replica load falls in
// that level (contiguous, since the level is nonincreasing in r).  cls < 0
// marks a candidate index outside [0, N).
struct CandInfo {
  int32_t cls, ti, rlo, rhi;
  int32_t cell, tp;  // cell index, TP degree (profiling cost per second)
  int32_t pad0, pad1;
};

// Per (order, candidate) constants of the exclusion scorer.  With H the
// (max,min) convolution of every class except the candidate's, U the best
// value reachable without the candidate's cell and f_r the ratio of r
// replicas on the candidate's cell, a scenario's objective is
//   tau = max(U, max_{r in [rlo, rhi]} min(f_r, H[G - t*r])).
struct TileInfo {
  int32_t cls, t, rlo, rhi;  // class, TP degree, replica range (rlo > rhi: unused cell)
  int32_t u_m, u_p;          // U of the conservative / optimistic realisation (bits)
  int32_t m_m, m_p;          // M at rlo, the largest over the range, of each realisation (bits; 0 when unused)
  int32_t state;             // 0 = solve, 1 = measured, -1 = invalid candidate
  int32_t cell;              // candidate cell index
  int32_t toff;              // option index of (class, TP, rlo): M and thresholds of the range
  int32_t pad;
};

// Workspace layout; every region is 256-byte aligned.
struct WsLayout {
  size_t bmap;     // int8  [K][G+1]   load level of r replicas (-1 = none)
  size_t cand;     // CandInfo [E]
  size_t base;     // int32 [O][2]     base tau bits (conservative, optimistic)
  size_t opts;     // float [O][2][K][PP][2] option (cap, tail), lane kernel only
  size_t partial;  // double [O][E][ceil(S/64)]
  size_t tiles;      // TileInfo [O][E]                       exclusion scorer
  size_t tabB;       // int32 [O][2][K][3][K][G] set-up tables when LDS is too small
  size_t mopt;       // int32 [O][2][K*P] M = H[G - t*r] of every option (class, TP, r)
  size_t thr;        // float [O][2][K*P] capacity threshold of every option
  size_t list;       // int4 [O * E] live tiles of every order, longest replica range first
  size_t btab;       // int32 [O][2][K][G] B tables of the general set-up
  size_t live;       // int32 [1] number of listed tiles
  size_t crec;       // [O][2] per-realisation results of the certificate under the whole objective
  size_t flag;     // int32 [4]        validation / error flags
  size_t total;
  int64_t n_partial;  // ceil(S / 64)
  int32_t pp;         // options per class of the lane kernel (0 if unused)
};

WsLayout ws_layout(const DevProblem &P, int64_t O, int64_t E, int64_t S);

// Static device scratch of fs_score_candidates_noalloc (FS_NOALLOC_SCRATCH_BYTES
// in the public header), and its address on the current device.
constexpr size_t kNoAllocScratchBytes = (size_t)32 << 20;
hipError_t scratch_address(void **ptr);

// Lane-per-scenario scoring supports these shapes.
bool lane_kernel_supported(const DevProblem &P);
int lane_kernel_options(int G);
// Exclusion scoring supports every problem without critical floors.
bool excl_kernel_supported(const DevProblem &P);

// ---- launchers (fs_kernels.hip) --------------------------------------------
struct ScoreArgs {
  const float *cap_lo, *cap_hi, *tail_lo, *tail_hi;
  const uint8_t *measured;
  const int32_t *cand;
  const float *cap_s, *tail_s;
  int32_t O, E, S;
  double *score, *gap_now;
  int32_t *best;
  float *tau_dump;
  uint8_t *ws;
  WsLayout L;
  int kernel;  // 1 = wave per scenario, 2 = lane per scenario, 3 = exclusion
  int spl;     // exclusion scorer: samples per lane (4, 8 or 16; 0 = default)
  int waves;   // exclusion scorer: wavefronts of its grid (0 = default)
  int setup;   // exclusion scorer set-up: 0 automatic, 1 general
  hipEvent_t ev_begin, ev_end;  // recorded around the scoring kernel launches if set
  int timing_launches;          // back-to-back launches of the scoring kernel between the events
  int thr_search;               // exclusion set-up: where the capacity-threshold search starts
                                // (0 window, 1 stepping, 2 bisection; identical results)
};

struct AllocOut {
  float *objective;
  uint8_t *tp_index;
  uint16_t *replicas;
  uint8_t *floors_met;
  float *goodput;
};

hipError_t launch_setup(const DevProblem &P, const int32_t *cand, int32_t E, uint8_t *ws,
                        const WsLayout &L, hipStream_t s);
hipError_t launch_score(const DevProblem &P, const ScoreArgs &a, hipStream_t s);
hipError_t launch_solve_batch(const DevProblem &P, const float *cap, const float *tail, int64_t n,
                              AllocOut out, uint8_t *ws, const WsLayout &L, hipStream_t s);
// The whole lexicographic objective (levels 1-4): LDS of a solve block with
// n_alloc allocations, and the launches.
size_t lds_bytes_lex(const DevProblem &P, int n_alloc);
constexpr size_t kLexLdsLimit = 64 * 1024;
hipError_t launch_solve_batch_lex(const DevProblem &P, const float *cap, const float *tail, int64_t n,
                                  AllocOut out, double *gp64, uint8_t *ws, const WsLayout &L, hipStream_t s);
// with_state false: only the orders' two records (for a caller that forms
// the gaps itself; state, gap_mm and gap_gp are then not written).
hipError_t launch_certify_lex(const DevProblem &P, const float *cap_lo, const float *cap_hi, const float *tail_lo,
                              const float *tail_hi, const uint8_t *measured, int32_t O, float eps, int32_t *state,
                              AllocOut cons, AllocOut opt, double *gap_mm, double *gap_gp, uint8_t *ws,
                              const WsLayout &L, hipStream_t s, bool with_state = true);
hipError_t launch_certify(const DevProblem &P, const float *cap_lo, const float *cap_hi,
                          const float *tail_lo, const float *tail_hi, const uint8_t *measured,
                          int32_t O, float eps, int32_t *state, AllocOut cons, AllocOut opt,
                          double *gap, uint8_t *ws, const WsLayout &L, hipStream_t s);
// ---- profiling loop (Algorithm 1) -------------------------------------------
// Device state of fs_profile_loop: a working copy of the intervals, this
// round's certificate and scores, the allocation each trajectory returns so
// far, and the caller's per-trajectory outputs.
struct LoopDev {
  float *cap_lo, *cap_hi, *tail_lo, *tail_hi;  // [O][N] working intervals
  uint8_t *measured;                           // [O][N]
  int32_t *cert_state;                         // [O] this round's certificate
  AllocOut cons;                               // [O] this round's conservative allocation
  AllocOut fin;                                // [O] the allocation returned so far
  double *score, *gap_now;                     // [O][E], [O] this round's scores
  int32_t *best;                               // [O]
  uint8_t *running;                            // [O] 1 while the trajectory continues
  int32_t *n_running;                          // [1] running trajectories (launch_loop_count)
  int32_t *state;                              // [O] caller outputs (fs_loop_out)
  uint8_t *finished;
  int32_t *rounds;
  double *gpu_seconds;
  int32_t *reveals;                            // [O][max_rounds] or NULL
  int32_t max_rounds;
};

// The goodput stage of the stage-wise score without full solves (problems
// without critical floors whose set-up fits): per (order, realisation)
// every option's (ratio, served rate) and the sorted distinct ratios, and
// per (order, realisation, class) and interval between them the knapsack
// of the other classes (G + 1 binary64) and the class's best options (4
// binary64).  fast = 0 when not available.
struct LexExclRegions {
  size_t opt, bp, nbp, V, W;
  int32_t nbmax;  // breakpoints per (order, realisation) at most: K x options per class + 1
  int fast;
};
LexExclRegions lex_excl_regions(const DevProblem &P, int64_t O, size_t *at);

// Workspace of fs_profile_loop: the scorer's layout, then the loop's own
// regions (offsets from the workspace start).
struct LoopLayout {
  WsLayout score;
  size_t cap_lo, cap_hi, tail_lo, tail_hi, measured, cert_state, cons_obj, cons_tp, cons_rep, cons_fm,
      cons_gp, fin_obj, fin_tp, fin_rep, fin_fm, fin_gp, scores, gap_now, best, running, n_running;
  size_t scores_gp, part_gp, gap_mm, gap_gp;  // the stage-wise score (whole objective)
  LexExclRegions lex_fast;
  size_t total;
};

LoopLayout loop_layout(const DevProblem &P, int64_t O, int64_t E, int64_t S);

// The stage-wise score under the whole objective: the scorer's layout plus a
// second array of partials, the order's two stages and a scratch state.
struct LexScoreLayout {
  WsLayout score;
  size_t part_gp, gap_mm, gap_gp, total;
  LexExclRegions fast;
};
LexScoreLayout lex_score_layout(const DevProblem &P, int64_t O, int64_t E, int64_t S);
// fast: the goodput stage without full solves where the layout has it (else
// every scenario is solved in full, as with fast = 0).  setup_here: build the
// bucket map and the candidate records in the call's first launch (else
// they are in the workspace already).  side, fork, join: a second stream
// and two events for the certificate solves (all three, or none).
hipError_t launch_score_lex(const DevProblem &P, const float *cap_lo, const float *cap_hi, const float *tail_lo,
                            const float *tail_hi, const uint8_t *measured, const int32_t *cand, const float *cap_s,
                            const float *tail_s, int32_t O, int32_t E, int32_t S, double *score_mm,
                            double *score_gp, double *gap_mm, double *gap_gp, int32_t *best, uint8_t *ws,
                            const LexScoreLayout &L, int fast, bool setup_here, hipStream_t s,
                            hipStream_t side = nullptr, hipEvent_t fork = nullptr, hipEvent_t join = nullptr);

// Interval refit and sample clamping (Algorithm 1's fit step).  The refit
// outputs may alias its inputs.
hipError_t launch_refit(const DevProblem &P, const float *cap_lo, const float *cap_hi, const float *tail_lo,
                        const float *tail_hi, const uint8_t *measured, int32_t O, float *cap_lo_out,
                        float *tail_lo_out, float *tail_hi_out, hipStream_t s);
hipError_t launch_clamp_samples(const DevProblem &P, const int32_t *cand, int32_t E, const float *cap_lo,
                                const float *cap_hi, const float *tail_lo, const float *tail_hi, const float *cap_s,
                                const float *tail_s, int32_t O, int32_t S, float *cs_out, float *ts_out,
                                hipStream_t s);
// Extra workspace of a loop with the fit step, after LoopLayout::total:
// refitted cap_lo, tail_lo, tail_hi [O][N] and clamped samples [O][E][S] x 2.
struct RefitLayout {
  size_t cap_lo, tail_lo, tail_hi, cap_s, tail_s, total;
};
RefitLayout refit_layout(const DevProblem &P, int64_t O, int64_t E, int64_t S, size_t start);
LoopDev loop_dev(const LoopLayout &L, uint8_t *ws, int64_t O);

hipError_t launch_loop_init(const LoopDev &L, int32_t O, hipStream_t s);
// After a certificate: trajectories that certified or have no unmeasured
// candidate end (their candidates are then marked measured, so the scorer
// skips them); every running trajectory takes A- as its allocation so far.
hipError_t launch_loop_decide(const DevProblem &P, const LoopDev &L, const int32_t *cand, int32_t E,
                              int32_t O, hipStream_t s);
// Counts the running trajectories into n_running.
hipError_t launch_loop_count(const LoopDev &L, int32_t O, hipStream_t s);
// Reveals one candidate of every running trajectory (policy 0: best[o],
// policy 1: the first unmeasured one of order[o]).
hipError_t launch_loop_reveal(const DevProblem &P, const LoopDev &L, const float *truth_cap,
                              const float *truth_tail, const int32_t *cand, int32_t E, int32_t O,
                              int32_t policy, const int32_t *order, hipStream_t s);
// Overwrites the working tail_lo with the measured-only table (unmeasured
// cells +inf, measured cells their point tails) for the final solve.
hipError_t launch_loop_measured_table(const DevProblem &P, const LoopDev &L, int32_t O, hipStream_t s);
// Copies the returned allocations out (A- of a certified trajectory, meas of
// one that ended undecided) and evaluates them on the true table.
hipError_t launch_loop_output(const DevProblem &P, const LoopDev &L, const AllocOut &meas, const uint8_t *ws,
                              const WsLayout &SL, const float *truth_cap, const float *truth_tail, int32_t O,
                              AllocOut out, float *tau_truth, hipStream_t s);

// ---- class policies with several metrics (Eq. 5 in full) -----------------------
constexpr int kMaxMetrics = 8;

struct DevPolicy {
  int32_t M;            // tail metrics per cell
  int32_t has_success;  // success floors given
  int32_t per_class;    // cells per class (NT * B)
  int32_t N;            // cells
  float limit[kMaxClasses * kMaxMetrics];  // [K][M]
  float success_min[kMaxClasses];
};

// out[j] = 0 if cell (j mod N) passes its class's policy, else +inf.
hipError_t launch_reduce_cells(const DevPolicy &Q, const float *tails, const float *success, int64_t rows,
                               float *out, hipStream_t s);
// out[o][e][s] = 0 if the sample passes the policy of cand[e]'s class, else +inf.
hipError_t launch_reduce_samples(const DevPolicy &Q, const int32_t *cand, int32_t E, const float *tail_s,
                                 const float *succ_s, int32_t O, int32_t S, float *out, hipStream_t s);

// Device-side input checks (FS_VALIDATE=1): flag[0] counts bad cell values,
// flag[1] candidate indices outside [0, N).  Zero the flags first.
hipError_t launch_zero_flags(int32_t *flag, hipStream_t s);
hipError_t launch_validate_cells(const float *cap, const float *tail, int64_t n, int32_t *flag,
                                 hipStream_t s);
hipError_t launch_validate_cands(const int32_t *cand, int32_t E, int32_t N, int32_t *flag, hipStream_t s);

}  // namespace fs
