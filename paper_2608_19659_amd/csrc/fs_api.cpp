// fs_api.cpp -- host side of libfleetsieve's C ABI (include/fleetsieve.h):
// argument validation, problem constants, workspace layout and kernel
// launches on the caller's stream.
#include "fleetsieve.h"

#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <utility>
#include <vector>

#include "fs_internal.h"

static_assert(fs::kNoAllocScratchBytes == FS_NOALLOC_SCRATCH_BYTES, "scratch size differs from the header");

struct fs_context {
  int device;
  int score_kernel;  // 0 auto, 1 wave per scenario, 2 lane per scenario, 3 exclusion
  int timing;        // back-to-back scoring-kernel launches between timing events (0 = off)
  int spl;           // exclusion scorer samples per lane (0 = default)
  int waves;         // exclusion scorer grid in wavefronts (0 = default)
  int setup;         // exclusion scorer set-up: 0 automatic, 1 general
  int loop_objective;  // profiling loop certificate: 0 max-min, 1 whole objective
  int loop_refit;      // profiling loop fit step: 0 off, 1 interval refit every round
  int thr_search;      // exclusion set-up: capacity-threshold search start (0 window, 1 stepping, 2 bisection)
  int32_t *pinned;   // pinned host word: running trajectories read back by fs_profile_loop
  void *scratch;     // this device's address of the static scratch of fs_score_candidates_noalloc
  // a second stream (default priority) and the fork / join events of the
  // stage-wise score
  hipStream_t side;
  hipEvent_t fork, join;
  struct Timed {
    hipEvent_t begin, end;
    int launches;
  };
  std::vector<Timed> events;
};

namespace {

thread_local std::string g_error;

fs_status fail(fs_status s, const std::string &msg) {
  g_error = msg;
  return s;
}

fs_status hip_fail(hipError_t e, const char *what) {
  return fail(FS_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

bool env_validate() {
  const char *v = std::getenv("FS_VALIDATE");
  return v && v[0] == '1';
}

// Checks the problem statement and fills the kernel-side constants.
fs_status make_problem(const fs_problem *p, fs::DevProblem *P) {
  if (!p) return fail(FS_ERR_INVALID_ARGUMENT, "problem is NULL");
  if (!p->tp || !p->levels || !p->demand || !p->slo)
    return fail(FS_ERR_INVALID_ARGUMENT, "problem arrays tp/levels/demand/slo must not be NULL");
  if (p->n_classes < 1 || p->n_classes > FS_MAX_CLASSES)
    return fail(FS_ERR_INVALID_ARGUMENT, "n_classes must be in [1, 64]");
  if (p->n_tp < 1 || p->n_tp > FS_MAX_TP) return fail(FS_ERR_INVALID_ARGUMENT, "n_tp must be in [1, 8]");
  if (p->n_levels < 1 || p->n_levels > FS_MAX_LEVELS)
    return fail(FS_ERR_INVALID_ARGUMENT, "n_levels must be in [1, 32]");
  if (p->budget < 1 || p->budget > FS_MAX_BUDGET)
    return fail(FS_ERR_INVALID_ARGUMENT, "budget must be in [1, 4096]");
  std::memset(P, 0, sizeof(*P));
  P->K = p->n_classes;
  P->NT = p->n_tp;
  P->B = p->n_levels;
  P->G = p->budget;
  P->N = P->K * P->NT * P->B;
  for (int t = 0; t < p->n_tp; ++t) {
    if (p->tp[t] < 1) return fail(FS_ERR_INVALID_ARGUMENT, "tp degrees must be >= 1");
    if (t > 0 && p->tp[t] <= p->tp[t - 1])
      return fail(FS_ERR_INVALID_ARGUMENT, "tp degrees must be strictly ascending");
    P->tp[t] = p->tp[t];
  }
  if (p->budget < p->tp[0]) return fail(FS_ERR_INVALID_ARGUMENT, "budget is below the smallest TP degree");
  P->optoff[0] = 0;
  for (int t = 0; t < p->n_tp; ++t) P->optoff[t + 1] = P->optoff[t] + p->budget / p->tp[t];
  for (int b = 0; b < p->n_levels; ++b) {
    const float v = p->levels[b];
    if (!(v > 0.0f) || !std::isfinite(v)) return fail(FS_ERR_INVALID_ARGUMENT, "levels must be finite and > 0");
    if (b > 0 && !(v > p->levels[b - 1]))
      return fail(FS_ERR_INVALID_ARGUMENT, "levels must be strictly ascending");
    P->levels[b] = v;
  }
  for (int i = 0; i < p->n_classes; ++i) {
    const float d = p->demand[i];
    if (!(d >= 0x1p-32f && d <= 0x1p32f)) return fail(FS_ERR_INVALID_ARGUMENT, "demand must be in [2^-32, 2^32]");
    if (std::isnan(p->slo[i])) return fail(FS_ERR_INVALID_ARGUMENT, "slo must not be NaN");
    P->demand[i] = d;
    P->slo[i] = p->slo[i];
    P->rcp_demand[i] = 1.0 / (double)d;
    if (p->floor_rps) {
      const float f = p->floor_rps[i];
      if (!(f >= 0.0f) || !std::isfinite(f))
        return fail(FS_ERR_INVALID_ARGUMENT, "floor_rps must be finite and >= 0");
      P->floor_rps[i] = f;
      if (f > 0.0f) P->has_floor = 1;
    }
  }
  return FS_OK;
}

struct DeviceGuard {
  int prev = -1;  // device to restore (-1: none, already current)
  hipError_t err = hipSuccess;
  explicit DeviceGuard(int dev) {
    err = hipGetDevice(&prev);
    if (err == hipSuccess && prev == dev) prev = -1;
    else if (err == hipSuccess) err = hipSetDevice(dev);
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

// FS_VALIDATE=1: wait for the flag words and turn them into a status.
fs_status read_flags(const fs::WsLayout &L, uint8_t *ws, hipStream_t s, const char *what) {
  int32_t flag[4] = {0, 0, 0, 0};
  hipError_t e = hipMemcpyAsync(flag, ws + L.flag, sizeof(flag), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, what);
  if (flag[0]) return fail(FS_ERR_INVALID_ARGUMENT, std::string(what) + ": " + std::to_string(flag[0]) +
                                                       " cell values out of range (capacity must be 0 or in "
                                                       "[2^-64, 2^64], tail >= 0 and not NaN)");
  if (flag[1]) return fail(FS_ERR_INVALID_ARGUMENT, std::string(what) + ": " + std::to_string(flag[1]) +
                                                       " candidate cell indices outside [0, N)");
  return FS_OK;
}

fs::AllocOut to_out(const fs_alloc &a) {
  return fs::AllocOut{a.objective, a.tp_index, a.replicas, a.floors_met, a.goodput};
}

}  // namespace

extern "C" {

const char *fs_last_error(void) { return g_error.c_str(); }

fs_status fs_context_create(int hip_device, fs_context **out) {
  if (!out) return fail(FS_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  int n = 0;
  hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess || n == 0) return fail(FS_ERR_DEVICE, "no HIP device available");
  if (hip_device < 0 || hip_device >= n) return fail(FS_ERR_INVALID_ARGUMENT, "hip_device out of range");
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, hip_device);
  if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(FS_ERR_UNSUPPORTED, std::string("libfleetsieve is built for gfx950, device is ") + prop.gcnArchName);
  int32_t *pinned = nullptr;
  e = hipSetDevice(hip_device);
  if (e == hipSuccess) e = hipHostMalloc((void **)&pinned, 64, hipHostMallocDefault);
  if (e != hipSuccess) return hip_fail(e, "hipHostMalloc");
  // the static scratch's address on this device (the device is current)
  void *scratch = nullptr;
  e = fs::scratch_address(&scratch);
  if (e != hipSuccess) {
    (void)hipHostFree(pinned);
    return hip_fail(e, "hipGetSymbolAddress(scratch)");
  }
  // the stage-wise score's second stream and its fork / join events
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  e = hipStreamCreateWithFlags(&side, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&fork, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&join, hipEventDisableTiming);
  if (e != hipSuccess) {
    if (fork) (void)hipEventDestroy(fork);
    if (side) (void)hipStreamDestroy(side);
    (void)hipHostFree(pinned);
    return hip_fail(e, "second stream of the stage-wise score");
  }
  *out = new fs_context{hip_device, 0, 0, 0, 0, 0, 0, 0, 0, pinned, scratch, side, fork, join, {}};
  return FS_OK;
}

void fs_context_destroy(fs_context *ctx) {
  if (!ctx) return;
  if (ctx->pinned) (void)hipHostFree(ctx->pinned);
  if (ctx->fork) (void)hipEventDestroy(ctx->fork);
  if (ctx->join) (void)hipEventDestroy(ctx->join);
  if (ctx->side) (void)hipStreamDestroy(ctx->side);
  for (auto &ev : ctx->events) {
    (void)hipEventDestroy(ev.begin);
    (void)hipEventDestroy(ev.end);
  }
  delete ctx;
}

fs_status fs_context_kernel_timing(fs_context *ctx, double *total_ms, int64_t *launches) {
  if (!ctx || !total_ms || !launches) return fail(FS_ERR_INVALID_ARGUMENT, "NULL argument");
  double sum = 0.0;
  int64_t n = 0;
  hipError_t err = hipSuccess;
  for (auto &ev : ctx->events) {
    float ms = 0.0f;
    hipError_t e = hipEventSynchronize(ev.end);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev.begin, ev.end);
    if (e != hipSuccess && err == hipSuccess) err = e;
    sum += ms;
    n += ev.launches;
    (void)hipEventDestroy(ev.begin);
    (void)hipEventDestroy(ev.end);
  }
  *launches = n;
  *total_ms = sum;
  ctx->events.clear();
  if (err != hipSuccess) return hip_fail(err, "kernel timing");
  return FS_OK;
}

fs_status fs_context_set_option(fs_context *ctx, fs_option option, int64_t value) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  if (option == FS_OPT_SCORE_KERNEL) {
    if (value < 0 || value > 3) return fail(FS_ERR_INVALID_ARGUMENT, "score kernel must be 0, 1, 2 or 3");
    ctx->score_kernel = (int)value;
    return FS_OK;
  }
  if (option == FS_OPT_SAMPLES_PER_LANE) {
    if (value != 0 && value != 4 && value != 8 && value != 16)
      return fail(FS_ERR_INVALID_ARGUMENT, "samples per lane must be 0, 4, 8 or 16");
    ctx->spl = (int)value;
    return FS_OK;
  }
  if (option == FS_OPT_SCORER_WAVES) {
    if (value < 0 || value > (1 << 20))
      return fail(FS_ERR_INVALID_ARGUMENT, "scorer wavefronts must be in [0, 2^20]");
    ctx->waves = (int)value;
    return FS_OK;
  }
  if (option == FS_OPT_LOOP_REFIT) {
    if (value != 0 && value != 1) return fail(FS_ERR_INVALID_ARGUMENT, "loop refit must be 0 or 1");
    ctx->loop_refit = (int)value;
    return FS_OK;
  }
  if (option == FS_OPT_LOOP_OBJECTIVE) {
    if (value != FS_OBJECTIVE_MAXMIN && value != FS_OBJECTIVE_LEXICOGRAPHIC)
      return fail(FS_ERR_INVALID_ARGUMENT, "loop objective must be FS_OBJECTIVE_MAXMIN or FS_OBJECTIVE_LEXICOGRAPHIC");
    ctx->loop_objective = (int)value;
    return FS_OK;
  }
  if (option == FS_OPT_THRESHOLD_SEARCH) {
    if (value < 0 || value > 2) return fail(FS_ERR_INVALID_ARGUMENT, "threshold search must be 0, 1 or 2");
    ctx->thr_search = (int)value;
    return FS_OK;
  }
  if (option == FS_OPT_SETUP) {
    if (value != 0 && value != 1) return fail(FS_ERR_INVALID_ARGUMENT, "set-up must be 0 or 1");
    ctx->setup = (int)value;
    return FS_OK;
  }
  if (option == FS_OPT_KERNEL_TIMING) {
    if (value < 0 || value > 64) return fail(FS_ERR_INVALID_ARGUMENT, "kernel timing must be in [0, 64]");
    ctx->timing = (int)value;
    return FS_OK;
  }
  return fail(FS_ERR_INVALID_ARGUMENT, "unknown option");
}

fs_status fs_validate_problem(const fs_problem *p) {
  fs::DevProblem P;
  return make_problem(p, &P);
}

fs_status fs_workspace_size(const fs_problem *p, int32_t n_orders, int32_t n_cand, int32_t n_samples,
                            size_t *bytes) {
  if (!bytes) return fail(FS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  if (n_orders < 0 || n_cand < 0 || n_samples < 0)
    return fail(FS_ERR_INVALID_ARGUMENT, "sizes must be >= 0");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  *bytes = fs::ws_layout(P, n_orders, n_cand, n_samples).total;
  return FS_OK;
}

fs_status fs_solve_batch(fs_context *ctx, const fs_problem *p, const float *d_cap, const float *d_tail,
                         int64_t n_scenarios, fs_alloc out, void *d_workspace, size_t workspace_bytes,
                         hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  if (n_scenarios < 0 || n_scenarios > 0x7fffffff)
    return fail(FS_ERR_INVALID_ARGUMENT, "n_scenarios must be in [0, 2^31)");
  if (n_scenarios > 0 && (!d_cap || !d_tail)) return fail(FS_ERR_INVALID_ARGUMENT, "cell arrays are NULL");
  const fs::WsLayout L = fs::ws_layout(P, 0, 0, 0);
  if (!d_workspace) return fail(FS_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (workspace_bytes < L.total)
    return fail(FS_ERR_WORKSPACE_TOO_SMALL, "workspace needs " + std::to_string(L.total) + " bytes");
  if (n_scenarios == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  uint8_t *ws = (uint8_t *)d_workspace;
  hipError_t e;
  if (env_validate()) {
    int32_t *flag = (int32_t *)(ws + L.flag);
    e = fs::launch_zero_flags(flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(d_cap, d_tail, n_scenarios * (int64_t)P.N, flag, stream);
    if (e != hipSuccess) return hip_fail(e, "validation launch");
    st = read_flags(L, ws, stream, "fs_solve_batch");
    if (st != FS_OK) return st;
  }
  e = fs::launch_setup(P, nullptr, 0, ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "set-up launch");
  e = fs::launch_solve_batch(P, d_cap, d_tail, n_scenarios, to_out(out), ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "solve launch");
  return FS_OK;
}

// Shared checks of the whole-objective calls: the stage's LDS must fit.
static fs_status lex_supported(const fs::DevProblem &P, int n_alloc) {
  const size_t need = fs::lds_bytes_lex(P, n_alloc);
  if (need > fs::kLexLdsLimit)
    return fail(FS_ERR_UNSUPPORTED, "the whole objective needs " + std::to_string(need) +
                                        " bytes of LDS for this problem (at most 65536: about (28 + 2 K)(G + 1) "
                                        "+ 1 KiB)");
  return FS_OK;
}

fs_status fs_solve_batch_lex(fs_context *ctx, const fs_problem *p, const float *d_cap, const float *d_tail,
                             int64_t n_scenarios, fs_alloc out, double *d_goodput64, void *d_workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  st = lex_supported(P, 1);
  if (st != FS_OK) return st;
  if (n_scenarios < 0 || n_scenarios > 0x7fffffff)
    return fail(FS_ERR_INVALID_ARGUMENT, "n_scenarios must be in [0, 2^31)");
  if (n_scenarios > 0 && (!d_cap || !d_tail)) return fail(FS_ERR_INVALID_ARGUMENT, "cell arrays are NULL");
  const fs::WsLayout L = fs::ws_layout(P, 0, 0, 0);
  if (!d_workspace) return fail(FS_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (workspace_bytes < L.total)
    return fail(FS_ERR_WORKSPACE_TOO_SMALL, "workspace needs " + std::to_string(L.total) + " bytes");
  if (n_scenarios == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  uint8_t *ws = (uint8_t *)d_workspace;
  hipError_t e;
  if (env_validate()) {
    int32_t *flag = (int32_t *)(ws + L.flag);
    e = fs::launch_zero_flags(flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(d_cap, d_tail, n_scenarios * (int64_t)P.N, flag, stream);
    if (e != hipSuccess) return hip_fail(e, "validation launch");
    st = read_flags(L, ws, stream, "fs_solve_batch_lex");
    if (st != FS_OK) return st;
  }
  e = fs::launch_setup(P, nullptr, 0, ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "set-up launch");
  e = fs::launch_solve_batch_lex(P, d_cap, d_tail, n_scenarios, to_out(out), d_goodput64, ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "solve launch");
  return FS_OK;
}

fs_status fs_score_lex_workspace_size(const fs_problem *p, int32_t n_orders, int32_t n_cand, int32_t n_samples,
                                      size_t *bytes) {
  if (!bytes) return fail(FS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  if (n_orders < 0 || n_cand < 0 || n_samples < 0) return fail(FS_ERR_INVALID_ARGUMENT, "sizes must be >= 0");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  *bytes = fs::lex_score_layout(P, n_orders, n_cand, n_cand > 0 ? n_samples : 0).total;
  return FS_OK;
}

fs_status fs_score_candidates_lex(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                                  const int32_t *d_cand, int32_t n_cand, const float *d_cap_s, const float *d_tail_s,
                                  int32_t n_samples, double *d_score_maxmin, double *d_score_goodput,
                                  double *d_gap_maxmin, double *d_gap_goodput, int32_t *d_best, void *d_workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  st = lex_supported(P, 2);
  if (st != FS_OK) return st;
  if (n_orders < 0 || n_orders > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_orders must be in [0, 65535]");
  if (n_cand < 0 || n_cand > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_cand must be in [0, 65535]");
  if (n_cand > 0 && (n_samples < 1 || n_samples > FS_MAX_SAMPLES))
    return fail(FS_ERR_INVALID_ARGUMENT, "n_samples must be in [1, 2^20]");
  if (n_orders > 0 && (!iv.cap_lo || !iv.cap_hi || !iv.tail_lo || !iv.tail_hi || !iv.measured))
    return fail(FS_ERR_INVALID_ARGUMENT, "interval arrays are NULL");
  if (n_orders > 0 && n_cand > 0 &&
      (!d_cand || !d_cap_s || !d_tail_s || !d_score_maxmin || !d_score_goodput))
    return fail(FS_ERR_INVALID_ARGUMENT, "candidate, sample or score arrays are NULL");
  const int32_t S = n_cand > 0 ? n_samples : 0;
  const fs::LexScoreLayout L = fs::lex_score_layout(P, n_orders, n_cand, S);
  if (!d_workspace) return fail(FS_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (workspace_bytes < L.total)
    return fail(FS_ERR_WORKSPACE_TOO_SMALL, "workspace needs " + std::to_string(L.total) + " bytes");
  if (n_orders == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  uint8_t *ws = (uint8_t *)d_workspace;
  // the bucket map and the candidate records in the call's first launch; the
  // goodput stage without full solves unless scoring kernel 1 (full solves)
  // is asked for
  hipError_t e = fs::launch_score_lex(P, iv.cap_lo, iv.cap_hi, iv.tail_lo, iv.tail_hi, iv.measured, d_cand, d_cap_s,
                                      d_tail_s, n_orders, n_cand, S, d_score_maxmin, d_score_goodput, d_gap_maxmin,
                                      d_gap_goodput, d_best, ws, L, ctx->score_kernel != 1, true, stream, ctx->side,
                                      ctx->fork, ctx->join);
  if (e != hipSuccess) return hip_fail(e, "stage-wise score launch");
  return FS_OK;
}

// fs_score_candidates and its variant without a workspace argument: with
// noalloc set, the workspace is the library's static device scratch, and
// neither the timing events (which create HIP events) nor the FS_VALIDATE
// read-back are used.
static fs_status score_candidates_impl(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                                       const int32_t *d_cand, int32_t n_cand, const float *d_cap_s,
                                       const float *d_tail_s, int32_t n_samples, double *d_score,
                                       double *d_gap_now, int32_t *d_best, float *d_tau_dump, void *d_workspace,
                                       size_t workspace_bytes, hipStream_t stream, bool noalloc) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  if (n_orders < 0 || n_orders > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_orders must be in [0, 65535]");
  if (n_cand < 0 || n_cand > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_cand must be in [0, 65535]");
  if (n_cand > 0 && (n_samples < 1 || n_samples > FS_MAX_SAMPLES))
    return fail(FS_ERR_INVALID_ARGUMENT, "n_samples must be in [1, 2^20]");
  int kernel = ctx->score_kernel;
  if (kernel == 0) kernel = fs::excl_kernel_supported(P) ? 3 : 1;
  if (kernel == 2 && !fs::lane_kernel_supported(P))
    return fail(FS_ERR_UNSUPPORTED,
                "lane-per-scenario scoring needs no floors, TP set {1,2,4,8} and budget 16, 32 or 64");
  if (kernel == 3 && !fs::excl_kernel_supported(P))
    return fail(FS_ERR_UNSUPPORTED, "exclusion scoring does not handle critical floors");
  if (kernel == 3 && (int64_t)n_orders * n_cand > INT32_MAX)
    return fail(FS_ERR_UNSUPPORTED, "exclusion scoring needs n_orders * n_cand < 2^31");
  const int32_t S = n_cand > 0 ? n_samples : 0;
  const fs::WsLayout L = fs::ws_layout(P, n_orders, n_cand, S);
  // the scratch limit depends on the sizes alone: checked before the arrays
  if (noalloc && L.total > workspace_bytes)
    return fail(FS_ERR_UNSUPPORTED, "these sizes need " + std::to_string(L.total) +
                                        " bytes of scratch; fs_score_candidates_noalloc has " +
                                        std::to_string(workspace_bytes) + " (use fs_score_candidates)");
  if (n_orders > 0 && (!iv.cap_lo || !iv.cap_hi || !iv.tail_lo || !iv.tail_hi || !iv.measured))
    return fail(FS_ERR_INVALID_ARGUMENT, "interval arrays are NULL");
  if (n_orders > 0 && n_cand > 0 && (!d_cand || !d_cap_s || !d_tail_s || !d_score))
    return fail(FS_ERR_INVALID_ARGUMENT, "candidate, sample or score arrays are NULL");
  if (noalloc) {
    if (!d_workspace) return fail(FS_ERR_INTERNAL, "the device scratch address is unknown");
  } else {
    if (!d_workspace) return fail(FS_ERR_INVALID_ARGUMENT, "workspace is NULL");
    if (workspace_bytes < L.total)
      return fail(FS_ERR_WORKSPACE_TOO_SMALL, "workspace needs " + std::to_string(L.total) + " bytes");
  }
  if (n_orders == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  uint8_t *ws = (uint8_t *)d_workspace;
  hipError_t e;
  if (!noalloc && env_validate()) {
    int32_t *flag = (int32_t *)(ws + L.flag);
    const int64_t cells = (int64_t)n_orders * P.N;
    e = fs::launch_zero_flags(flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(iv.cap_lo, iv.tail_lo, cells, flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(iv.cap_hi, iv.tail_hi, cells, flag, stream);
    if (e == hipSuccess && n_cand > 0)
      e = fs::launch_validate_cells(d_cap_s, d_tail_s, (int64_t)n_orders * n_cand * S, flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cands(d_cand, n_cand, P.N, flag, stream);
    if (e != hipSuccess) return hip_fail(e, "validation launch");
    st = read_flags(L, ws, stream, "fs_score_candidates");
    if (st != FS_OK) return st;
  }
  if (kernel != 3) {
    e = fs::launch_setup(P, d_cand, n_cand, ws, L, stream);
    if (e != hipSuccess) return hip_fail(e, "set-up launch");
  }
  fs::ScoreArgs a{iv.cap_lo, iv.cap_hi, iv.tail_lo, iv.tail_hi, iv.measured, d_cand, d_cap_s, d_tail_s,
                  n_orders, n_cand, S, d_score, d_gap_now, d_best, d_tau_dump, ws, L, kernel,
                  ctx->spl, ctx->waves, ctx->setup, nullptr, nullptr, 1, ctx->thr_search};
  if (!noalloc && ctx->timing && n_cand > 0) {
    e = hipEventCreate(&a.ev_begin);
    if (e == hipSuccess) e = hipEventCreate(&a.ev_end);
    if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
    a.timing_launches = ctx->timing;
    ctx->events.push_back({a.ev_begin, a.ev_end, ctx->timing});
  }
  e = fs::launch_score(P, a, stream);
  if (e != hipSuccess) return hip_fail(e, "score launch");
  return FS_OK;
}

fs_status fs_score_candidates(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                              const int32_t *d_cand, int32_t n_cand, const float *d_cap_s,
                              const float *d_tail_s, int32_t n_samples, double *d_score,
                              double *d_gap_now, int32_t *d_best, float *d_tau_dump, void *d_workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  return score_candidates_impl(ctx, p, iv, n_orders, d_cand, n_cand, d_cap_s, d_tail_s, n_samples, d_score,
                               d_gap_now, d_best, d_tau_dump, d_workspace, workspace_bytes, stream, false);
}

fs_status fs_score_candidates_noalloc(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                                      const int32_t *d_cand, int32_t n_cand, const float *d_cap_s,
                                      const float *d_tail_s, int32_t n_samples, double *d_score,
                                      double *d_gap_now, int32_t *d_best, float *d_tau_dump,
                                      hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  return score_candidates_impl(ctx, p, iv, n_orders, d_cand, n_cand, d_cap_s, d_tail_s, n_samples, d_score,
                               d_gap_now, d_best, d_tau_dump, ctx->scratch, fs::kNoAllocScratchBytes, stream,
                               true);
}

fs_status fs_loop_workspace_size(const fs_problem *p, int32_t n_orders, int32_t n_cand, int32_t n_samples,
                                 size_t *bytes) {
  if (!bytes) return fail(FS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  if (n_orders < 0 || n_cand < 0 || n_samples < 0) return fail(FS_ERR_INVALID_ARGUMENT, "sizes must be >= 0");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  *bytes = fs::loop_layout(P, n_orders, n_cand, n_cand > 0 ? n_samples : 0).total;
  return FS_OK;
}

fs_status fs_loop_refit_workspace_size(const fs_problem *p, int32_t n_orders, int32_t n_cand, int32_t n_samples,
                                       size_t *bytes) {
  if (!bytes) return fail(FS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  if (n_orders < 0 || n_cand < 0 || n_samples < 0) return fail(FS_ERR_INVALID_ARGUMENT, "sizes must be >= 0");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  const int32_t S = n_cand > 0 ? n_samples : 0;
  const size_t base = fs::loop_layout(P, n_orders, n_cand, S).total;
  *bytes = fs::refit_layout(P, n_orders, n_cand, S, base).total;
  return FS_OK;
}

fs_status fs_refit_intervals(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                             float *d_cap_lo_out, float *d_tail_lo_out, float *d_tail_hi_out, hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  if (n_orders < 0 || n_orders > 0x7fffffff) return fail(FS_ERR_INVALID_ARGUMENT, "n_orders must be >= 0");
  if (n_orders > 0 && (!iv.cap_lo || !iv.cap_hi || !iv.tail_lo || !iv.tail_hi || !iv.measured))
    return fail(FS_ERR_INVALID_ARGUMENT, "interval arrays are NULL");
  if (n_orders > 0 && (!d_cap_lo_out || !d_tail_lo_out || !d_tail_hi_out))
    return fail(FS_ERR_INVALID_ARGUMENT, "output arrays are NULL");
  if (n_orders == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  const hipError_t e = fs::launch_refit(P, iv.cap_lo, iv.cap_hi, iv.tail_lo, iv.tail_hi, iv.measured, n_orders,
                                        d_cap_lo_out, d_tail_lo_out, d_tail_hi_out, stream);
  if (e != hipSuccess) return hip_fail(e, "refit launch");
  return FS_OK;
}

fs_status fs_clamp_samples(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                           const int32_t *d_cand, int32_t n_cand, const float *d_cap_s, const float *d_tail_s,
                           int32_t n_samples, float *d_cap_out, float *d_tail_out, hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  if (n_orders < 0 || n_orders > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_orders must be in [0, 65535]");
  if (n_cand < 0 || n_cand > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_cand must be in [0, 65535]");
  if (n_samples < 0 || n_samples > FS_MAX_SAMPLES)
    return fail(FS_ERR_INVALID_ARGUMENT, "n_samples must be in [0, 2^20]");
  const int64_t n = (int64_t)n_orders * n_cand * n_samples;
  if (n > 0 && (!iv.cap_lo || !iv.cap_hi || !iv.tail_lo || !iv.tail_hi))
    return fail(FS_ERR_INVALID_ARGUMENT, "interval arrays are NULL");
  if (n > 0 && (!d_cand || !d_cap_s || !d_tail_s || !d_cap_out || !d_tail_out))
    return fail(FS_ERR_INVALID_ARGUMENT, "candidate, sample or output arrays are NULL");
  if (n == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  const hipError_t e = fs::launch_clamp_samples(P, d_cand, n_cand, iv.cap_lo, iv.cap_hi, iv.tail_lo, iv.tail_hi,
                                                d_cap_s, d_tail_s, n_orders, n_samples, d_cap_out, d_tail_out,
                                                stream);
  if (e != hipSuccess) return hip_fail(e, "clamp launch");
  return FS_OK;
}

fs_status fs_profile_loop(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders,
                          const float *d_truth_cap, const float *d_truth_tail, const int32_t *d_cand,
                          int32_t n_cand, const float *d_cap_s, const float *d_tail_s, int32_t n_samples,
                          float eps, fs_policy policy, const int32_t *d_order, int32_t max_rounds,
                          int32_t check_every, fs_loop_out out, void *d_workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  if (n_orders < 0 || n_orders > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_orders must be in [0, 65535]");
  if (n_cand < 0 || n_cand > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_cand must be in [0, 65535]");
  if (max_rounds < 0 || max_rounds > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "max_rounds must be in [0, 65535]");
  if (check_every < 0) return fail(FS_ERR_INVALID_ARGUMENT, "check_every must be >= 0");
  if (std::isnan(eps)) return fail(FS_ERR_INVALID_ARGUMENT, "eps must not be NaN");
  if (policy != FS_POLICY_SCORE && policy != FS_POLICY_ORDER)
    return fail(FS_ERR_INVALID_ARGUMENT, "policy must be FS_POLICY_SCORE or FS_POLICY_ORDER");
  if (policy == FS_POLICY_SCORE && n_cand > 0 && (n_samples < 1 || n_samples > FS_MAX_SAMPLES))
    return fail(FS_ERR_INVALID_ARGUMENT, "n_samples must be in [1, 2^20]");
  int kernel = ctx->score_kernel;
  if (kernel == 0) kernel = fs::excl_kernel_supported(P) ? 3 : 1;
  if (kernel == 2 && !fs::lane_kernel_supported(P))
    return fail(FS_ERR_UNSUPPORTED,
                "lane-per-scenario scoring needs no floors, TP set {1,2,4,8} and budget 16, 32 or 64");
  if (kernel == 3 && !fs::excl_kernel_supported(P))
    return fail(FS_ERR_UNSUPPORTED, "exclusion scoring does not handle critical floors");
  // the exclusion scorer's work list indexes (order, candidate) pairs in int32
  if (kernel == 3 && policy == FS_POLICY_SCORE && (int64_t)n_orders * n_cand > INT32_MAX)
    return fail(FS_ERR_UNSUPPORTED, "exclusion scoring needs n_orders * n_cand < 2^31");
  if (n_orders > 0 && (!iv.cap_lo || !iv.cap_hi || !iv.tail_lo || !iv.tail_hi || !iv.measured))
    return fail(FS_ERR_INVALID_ARGUMENT, "interval arrays are NULL");
  if (n_orders > 0 && (!d_truth_cap || !d_truth_tail))
    return fail(FS_ERR_INVALID_ARGUMENT, "true tables are NULL");
  if (n_orders > 0 && n_cand > 0 && !d_cand) return fail(FS_ERR_INVALID_ARGUMENT, "candidates are NULL");
  if (n_orders > 0 && n_cand > 0 && policy == FS_POLICY_SCORE && (!d_cap_s || !d_tail_s))
    return fail(FS_ERR_INVALID_ARGUMENT, "sample arrays are NULL");
  if (n_orders > 0 && n_cand > 0 && policy == FS_POLICY_ORDER && !d_order)
    return fail(FS_ERR_INVALID_ARGUMENT, "the reveal order is NULL");
  if (n_orders > 0 && (!out.state || !out.finished || !out.rounds || !out.gpu_seconds))
    return fail(FS_ERR_INVALID_ARGUMENT, "state, finished, rounds and gpu_seconds outputs are required");
  const bool lex = ctx->loop_objective == FS_OBJECTIVE_LEXICOGRAPHIC;
  if (lex) {
    st = lex_supported(P, 2);
    if (st != FS_OK) return st;
  }
  const int32_t S = (n_cand > 0 && policy == FS_POLICY_SCORE) ? n_samples : 0;
  const fs::LoopLayout LL = fs::loop_layout(P, n_orders, n_cand, S);
  const bool refit = ctx->loop_refit != 0;
  const fs::RefitLayout RL = fs::refit_layout(P, n_orders, n_cand, S, LL.total);
  const size_t need = refit ? RL.total : LL.total;
  if (!d_workspace) return fail(FS_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (workspace_bytes < need)
    return fail(FS_ERR_WORKSPACE_TOO_SMALL, "workspace needs " + std::to_string(need) + " bytes" +
                                                (refit ? " (fs_loop_refit_workspace_size)" : ""));
  if (n_orders == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  uint8_t *ws = (uint8_t *)d_workspace;
  hipError_t e;
  if (env_validate()) {
    int32_t *flag = (int32_t *)(ws + LL.score.flag);
    const int64_t cells = (int64_t)n_orders * P.N;
    e = fs::launch_zero_flags(flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(iv.cap_lo, iv.tail_lo, cells, flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(iv.cap_hi, iv.tail_hi, cells, flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(d_truth_cap, d_truth_tail, cells, flag, stream);
    if (e == hipSuccess && S > 0)
      e = fs::launch_validate_cells(d_cap_s, d_tail_s, (int64_t)n_orders * n_cand * S, flag, stream);
    if (e == hipSuccess && n_cand > 0) e = fs::launch_validate_cands(d_cand, n_cand, P.N, flag, stream);
    if (e != hipSuccess) return hip_fail(e, "validation launch");
    st = read_flags(LL.score, ws, stream, "fs_profile_loop");
    if (st != FS_OK) return st;
  }
  fs::LoopDev D = fs::loop_dev(LL, ws, n_orders);
  D.state = out.state;
  D.finished = out.finished;
  D.rounds = out.rounds;
  D.gpu_seconds = out.gpu_seconds;
  D.reveals = out.reveals;
  D.max_rounds = max_rounds;
  const size_t cells = (size_t)n_orders * P.N;
  e = hipMemcpyAsync(D.cap_lo, iv.cap_lo, 4 * cells, hipMemcpyDeviceToDevice, stream);
  if (e == hipSuccess) e = hipMemcpyAsync(D.cap_hi, iv.cap_hi, 4 * cells, hipMemcpyDeviceToDevice, stream);
  if (e == hipSuccess) e = hipMemcpyAsync(D.tail_lo, iv.tail_lo, 4 * cells, hipMemcpyDeviceToDevice, stream);
  if (e == hipSuccess) e = hipMemcpyAsync(D.tail_hi, iv.tail_hi, 4 * cells, hipMemcpyDeviceToDevice, stream);
  if (e == hipSuccess) e = hipMemcpyAsync(D.measured, iv.measured, cells, hipMemcpyDeviceToDevice, stream);
  if (e != hipSuccess) return hip_fail(e, "interval copy");
  e = fs::launch_setup(P, d_cand, n_cand, ws, LL.score, stream);
  if (e == hipSuccess) e = fs::launch_loop_init(D, n_orders, stream);
  if (e != hipSuccess) return hip_fail(e, "loop set-up launch");
  const fs::AllocOut none{nullptr, nullptr, nullptr, nullptr, nullptr};
  // With the fit step, the trajectories' own intervals (D.*) keep the initial
  // ones with the revealed cells collapsed; every round the certificate and
  // the score see their refit (R_*) and the samples clamped into it.
  float *R_cap_lo = refit ? (float *)(ws + RL.cap_lo) : D.cap_lo;
  float *R_tail_lo = refit ? (float *)(ws + RL.tail_lo) : D.tail_lo;
  float *R_tail_hi = refit ? (float *)(ws + RL.tail_hi) : D.tail_hi;
  float *R_cap_s = refit ? (float *)(ws + RL.cap_s) : nullptr;
  float *R_tail_s = refit ? (float *)(ws + RL.tail_s) : nullptr;
  for (int32_t rnd = 0; rnd <= max_rounds; ++rnd) {
    if (refit) {
      e = fs::launch_refit(P, D.cap_lo, D.cap_hi, D.tail_lo, D.tail_hi, D.measured, n_orders, R_cap_lo, R_tail_lo,
                           R_tail_hi, stream);
      if (e != hipSuccess) return hip_fail(e, "loop refit launch");
    }
    e = lex ? fs::launch_certify_lex(P, R_cap_lo, D.cap_hi, R_tail_lo, R_tail_hi, D.measured, n_orders, eps,
                                     D.cert_state, D.cons, none, nullptr, nullptr, ws, LL.score, stream)
            : fs::launch_certify(P, R_cap_lo, D.cap_hi, R_tail_lo, R_tail_hi, D.measured, n_orders, eps,
                                 D.cert_state, D.cons, none, nullptr, ws, LL.score, stream);
    if (e == hipSuccess) e = fs::launch_loop_decide(P, D, d_cand, n_cand, n_orders, stream);
    if (e != hipSuccess) return hip_fail(e, "loop certificate launch");
    if (rnd == max_rounds) break;
    if (check_every > 0 && rnd > 0 && rnd % check_every == 0) {
      e = fs::launch_loop_count(D, n_orders, stream);
      if (e == hipSuccess)
        e = hipMemcpyAsync(ctx->pinned, D.n_running, sizeof(int32_t), hipMemcpyDeviceToHost, stream);
      if (e == hipSuccess) e = hipStreamSynchronize(stream);
      if (e != hipSuccess) return hip_fail(e, "loop progress read-back");
      if (*ctx->pinned == 0) break;
    }
    if (policy == FS_POLICY_SCORE && n_cand > 0) {
      const float *cs = d_cap_s, *ts = d_tail_s;
      if (refit) {
        e = fs::launch_clamp_samples(P, d_cand, n_cand, R_cap_lo, D.cap_hi, R_tail_lo, R_tail_hi, d_cap_s,
                                     d_tail_s, n_orders, S, R_cap_s, R_tail_s, stream);
        if (e != hipSuccess) return hip_fail(e, "loop sample clamp launch");
        cs = R_cap_s;
        ts = R_tail_s;
      }
      if (lex) {  // the stage-wise score: the max-min stage first, then the goodput stage
        fs::LexScoreLayout XL{};
        XL.score = LL.score;
        XL.part_gp = LL.part_gp;
        XL.gap_mm = LL.gap_mm;
        XL.gap_gp = LL.gap_gp;
        XL.fast = LL.lex_fast;
        e = fs::launch_score_lex(P, R_cap_lo, D.cap_hi, R_tail_lo, R_tail_hi, D.measured, d_cand, cs, ts, n_orders,
                                 n_cand, S, D.score, (double *)(ws + LL.scores_gp), nullptr, nullptr, D.best, ws, XL,
                                 ctx->score_kernel != 1, false, stream);
      } else {
        fs::ScoreArgs a{R_cap_lo, D.cap_hi, R_tail_lo, R_tail_hi, D.measured, d_cand, cs, ts,
                        n_orders, n_cand, S, D.score, D.gap_now, D.best, nullptr, ws, LL.score, kernel,
                        ctx->spl, ctx->waves, ctx->setup, nullptr, nullptr, 1, ctx->thr_search};
        e = fs::launch_score(P, a, stream);
      }
      if (e != hipSuccess) return hip_fail(e, "loop score launch");
    }
    e = fs::launch_loop_reveal(P, D, d_truth_cap, d_truth_tail, d_cand, n_cand, n_orders, (int32_t)policy,
                               d_order, stream);
    if (e != hipSuccess) return hip_fail(e, "loop reveal launch");
  }
  // Algorithm 1's last line for the trajectories that ended undecided: the
  // best allocation over measured cells only, into this round's (no longer
  // needed) conservative allocation
  e = fs::launch_loop_measured_table(P, D, n_orders, stream);
  if (e == hipSuccess)
    e = lex ? fs::launch_solve_batch_lex(P, D.cap_lo, D.tail_lo, n_orders, D.cons, nullptr, ws, LL.score, stream)
            : fs::launch_solve_batch(P, D.cap_lo, D.tail_lo, n_orders, D.cons, ws, LL.score, stream);
  if (e == hipSuccess)
    e = fs::launch_loop_output(P, D, D.cons, ws, LL.score, d_truth_cap, d_truth_tail, n_orders,
                               to_out(out.final_alloc), out.tau_truth, stream);
  if (e == hipSuccess && out.tau_oracle)
    e = fs::launch_solve_batch(P, d_truth_cap, d_truth_tail, n_orders,
                               fs::AllocOut{out.tau_oracle, nullptr, nullptr, nullptr, nullptr}, ws, LL.score,
                               stream);
  if (e != hipSuccess) return hip_fail(e, "loop output launch");
  return FS_OK;
}

// Checks a policy and fills its kernel-side form.
static fs_status make_policy(const fs::DevProblem &P, const fs_slo_policy *pol, fs::DevPolicy *Q) {
  if (!pol) return fail(FS_ERR_INVALID_ARGUMENT, "policy is NULL");
  if (pol->n_metrics < 1 || pol->n_metrics > FS_MAX_METRICS)
    return fail(FS_ERR_INVALID_ARGUMENT, "n_metrics must be in [1, 8]");
  if (!pol->limit) return fail(FS_ERR_INVALID_ARGUMENT, "policy limits are NULL");
  std::memset(Q, 0, sizeof(*Q));
  Q->M = pol->n_metrics;
  Q->per_class = P.NT * P.B;
  Q->N = P.N;
  for (int i = 0; i < P.K * Q->M; ++i) {
    if (std::isnan(pol->limit[i])) return fail(FS_ERR_INVALID_ARGUMENT, "policy limits must not be NaN");
    Q->limit[i] = pol->limit[i];
  }
  if (pol->success_min) {
    Q->has_success = 1;
    for (int i = 0; i < P.K; ++i) {
      if (std::isnan(pol->success_min[i])) return fail(FS_ERR_INVALID_ARGUMENT, "success floors must not be NaN");
      Q->success_min[i] = pol->success_min[i];
    }
  }
  return FS_OK;
}

fs_status fs_reduce_cells(fs_context *ctx, const fs_problem *p, const fs_slo_policy *pol, const float *d_tails,
                          const float *d_success, int64_t n_rows, float *d_out, hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  fs::DevPolicy Q;
  st = make_policy(P, pol, &Q);
  if (st != FS_OK) return st;
  if (n_rows < 0 || n_rows > (int64_t)1 << 40) return fail(FS_ERR_INVALID_ARGUMENT, "n_rows out of range");
  if (n_rows > 0 && (!d_tails || !d_out)) return fail(FS_ERR_INVALID_ARGUMENT, "tail or output array is NULL");
  if (n_rows > 0 && Q.has_success && !d_success)
    return fail(FS_ERR_INVALID_ARGUMENT, "the policy has success floors but the success array is NULL");
  if (n_rows == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  const hipError_t e = fs::launch_reduce_cells(Q, d_tails, d_success, n_rows, d_out, stream);
  if (e != hipSuccess) return hip_fail(e, "reduce launch");
  return FS_OK;
}

fs_status fs_reduce_samples(fs_context *ctx, const fs_problem *p, const fs_slo_policy *pol, const int32_t *d_cand,
                            int32_t n_cand, const float *d_tail_s, const float *d_succ_s, int32_t n_orders,
                            int32_t n_samples, float *d_out, hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  fs::DevPolicy Q;
  st = make_policy(P, pol, &Q);
  if (st != FS_OK) return st;
  if (n_orders < 0 || n_orders > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_orders must be in [0, 65535]");
  if (n_cand < 0 || n_cand > 65535) return fail(FS_ERR_INVALID_ARGUMENT, "n_cand must be in [0, 65535]");
  if (n_samples < 0 || n_samples > FS_MAX_SAMPLES)
    return fail(FS_ERR_INVALID_ARGUMENT, "n_samples must be in [0, FS_MAX_SAMPLES]");
  const int64_t n = (int64_t)n_orders * n_cand * n_samples;
  if (n > 0 && (!d_cand || !d_tail_s || !d_out))
    return fail(FS_ERR_INVALID_ARGUMENT, "candidate, sample or output array is NULL");
  if (n > 0 && Q.has_success && !d_succ_s)
    return fail(FS_ERR_INVALID_ARGUMENT, "the policy has success floors but the success samples are NULL");
  if (n == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  const hipError_t e =
      fs::launch_reduce_samples(Q, d_cand, n_cand, d_tail_s, d_succ_s, n_orders, n_samples, d_out, stream);
  if (e != hipSuccess) return hip_fail(e, "reduce launch");
  return FS_OK;
}

fs_status fs_certify(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders, float eps,
                     int32_t *d_state, fs_alloc cons, fs_alloc opt, double *d_gap, void *d_workspace,
                     size_t workspace_bytes, hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  if (n_orders < 0 || n_orders > 0x7fffffff) return fail(FS_ERR_INVALID_ARGUMENT, "n_orders must be >= 0");
  if (std::isnan(eps)) return fail(FS_ERR_INVALID_ARGUMENT, "eps must not be NaN");
  if (n_orders > 0 && (!iv.cap_lo || !iv.cap_hi || !iv.tail_lo || !iv.tail_hi || !iv.measured || !d_state))
    return fail(FS_ERR_INVALID_ARGUMENT, "interval or state arrays are NULL");
  const fs::WsLayout L = fs::ws_layout(P, 0, 0, 0);
  if (!d_workspace) return fail(FS_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (workspace_bytes < L.total)
    return fail(FS_ERR_WORKSPACE_TOO_SMALL, "workspace needs " + std::to_string(L.total) + " bytes");
  if (n_orders == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  uint8_t *ws = (uint8_t *)d_workspace;
  hipError_t e;
  if (env_validate()) {
    int32_t *flag = (int32_t *)(ws + L.flag);
    const int64_t cells = (int64_t)n_orders * P.N;
    e = fs::launch_zero_flags(flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(iv.cap_lo, iv.tail_lo, cells, flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(iv.cap_hi, iv.tail_hi, cells, flag, stream);
    if (e != hipSuccess) return hip_fail(e, "validation launch");
    st = read_flags(L, ws, stream, "fs_certify");
    if (st != FS_OK) return st;
  }
  e = fs::launch_setup(P, nullptr, 0, ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "set-up launch");
  e = fs::launch_certify(P, iv.cap_lo, iv.cap_hi, iv.tail_lo, iv.tail_hi, iv.measured, n_orders, eps,
                         d_state, to_out(cons), to_out(opt), d_gap, ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "certify launch");
  return FS_OK;
}

fs_status fs_certify_lex(fs_context *ctx, const fs_problem *p, fs_intervals iv, int32_t n_orders, float eps,
                         int32_t *d_state, fs_alloc cons, fs_alloc opt, double *d_gap_maxmin,
                         double *d_gap_goodput, void *d_workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!ctx) return fail(FS_ERR_INVALID_ARGUMENT, "context is NULL");
  fs::DevProblem P;
  fs_status st = make_problem(p, &P);
  if (st != FS_OK) return st;
  st = lex_supported(P, 2);
  if (st != FS_OK) return st;
  if (n_orders < 0 || n_orders > 0x7fffffff) return fail(FS_ERR_INVALID_ARGUMENT, "n_orders must be >= 0");
  if (std::isnan(eps)) return fail(FS_ERR_INVALID_ARGUMENT, "eps must not be NaN");
  if (n_orders > 0 && (!iv.cap_lo || !iv.cap_hi || !iv.tail_lo || !iv.tail_hi || !iv.measured || !d_state))
    return fail(FS_ERR_INVALID_ARGUMENT, "interval or state arrays are NULL");
  const fs::WsLayout L = fs::ws_layout(P, 0, 0, 0);
  if (!d_workspace) return fail(FS_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (workspace_bytes < L.total)
    return fail(FS_ERR_WORKSPACE_TOO_SMALL, "workspace needs " + std::to_string(L.total) + " bytes");
  if (n_orders == 0) return FS_OK;
  DeviceGuard dg(ctx->device);
  if (dg.err != hipSuccess) return hip_fail(dg.err, "hipSetDevice");
  uint8_t *ws = (uint8_t *)d_workspace;
  hipError_t e;
  if (env_validate()) {
    int32_t *flag = (int32_t *)(ws + L.flag);
    const int64_t cells = (int64_t)n_orders * P.N;
    e = fs::launch_zero_flags(flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(iv.cap_lo, iv.tail_lo, cells, flag, stream);
    if (e == hipSuccess) e = fs::launch_validate_cells(iv.cap_hi, iv.tail_hi, cells, flag, stream);
    if (e != hipSuccess) return hip_fail(e, "validation launch");
    st = read_flags(L, ws, stream, "fs_certify_lex");
    if (st != FS_OK) return st;
  }
  e = fs::launch_setup(P, nullptr, 0, ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "set-up launch");
  e = fs::launch_certify_lex(P, iv.cap_lo, iv.cap_hi, iv.tail_lo, iv.tail_hi, iv.measured, n_orders, eps, d_state,
                             to_out(cons), to_out(opt), d_gap_maxmin, d_gap_goodput, ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "certify launch");
  return FS_OK;
}

}  // extern "C"
