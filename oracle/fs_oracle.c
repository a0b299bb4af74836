/*
 * fs_oracle.c -- plain, slow CPU oracle for FleetSieve (see fs_oracle.h).
 *
 * TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the
 * CPU-baseline leg of bench.py.  The product path never includes, links or
 * calls it, and it shares no code with the GPU path.
 *
 * What it computes, and where the paper defines it:
 *   - the fleet allocation of Section 3, Eq. (1)-(5): one homogeneous
 *     configuration (TP degree, replica count) per class, total GPUs within
 *     the budget G (Eq. 3), served load bounded by replica capacity and by
 *     demand (Eq. 2, 4), and a configuration usable only when its tail metric
 *     is within the class SLO (Eq. 5);
 *   - the lexicographic objective stated after Eq. (5): (1) critical floors
 *     whenever they can be met, (2) maximise the minimum satisfaction ratio
 *     r_i = x_i / lambda_i; ties go to fewer GPUs, then to the
 *     lexicographically smaller TP vector (the solvers orc_solve_*); and the
 *     whole objective with (3) maximum served goodput and (4) fewest GPUs
 *     (orc_solve_lex*, orc_certify_lex);
 *   - the conservative / optimistic realisations of Section 4.1;
 *   - the three-state certificate of Section 4.2;
 *   - the acquisition score of Section 4.3, score(e) = E[Gamma_t -
 *     Gamma_{t+1} | e], estimated over caller-supplied samples, with the
 *     profiling cost (duration x GPUs, Section 5) as strict tie-breaker.
 *
 * Fulfillment arithmetic is binary32 with one multiply and one divide per
 * option; no fused multiply-add (build with -ffp-contract=off).
 */
#include "fs_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
  int t_idx; /* index into tp[] */
  int r;     /* replicas        */
  int cost;  /* tp[t_idx] * r   */
  int cell;  /* cell(i, t_idx, bucket(i, r)) */
} orc_option;

static int orc_n_cells(const orc_problem *p) { return p->n_classes * p->n_tp * p->n_levels; }

static int orc_cell(const orc_problem *p, int i, int t, int b) {
  return (i * p->n_tp + t) * p->n_levels + b;
}

static int orc_is_critical(const orc_problem *p, int i) {
  return p->floor_rps != NULL && p->floor_rps[i] > 0.0f;
}

static int orc_has_critical(const orc_problem *p) {
  for (int i = 0; i < p->n_classes; ++i)
    if (orc_is_critical(p, i)) return 1;
  return 0;
}

int orc_check_problem(const orc_problem *p) {
  if (!p || !p->tp || !p->levels || !p->demand || !p->slo) return -1;
  if (p->n_classes < 1 || p->n_classes > ORC_MAX_CLASSES) return -1;
  if (p->n_tp < 1 || p->n_tp > ORC_MAX_TP) return -1;
  if (p->n_levels < 1 || p->n_levels > ORC_MAX_LEVELS) return -1;
  if (p->budget < 1 || p->budget > ORC_MAX_BUDGET) return -1;
  for (int t = 0; t < p->n_tp; ++t) {
    if (p->tp[t] < 1) return -1;
    if (t > 0 && p->tp[t] <= p->tp[t - 1]) return -1;
  }
  if (p->budget < p->tp[0]) return -1;
  for (int b = 0; b < p->n_levels; ++b) {
    if (!(p->levels[b] > 0.0f) || !isfinite(p->levels[b])) return -1;
    if (b > 0 && !(p->levels[b] > p->levels[b - 1])) return -1;
  }
  for (int i = 0; i < p->n_classes; ++i) {
    if (!(p->demand[i] > 0.0f) || !isfinite(p->demand[i])) return -1;
    if (isnan(p->slo[i])) return -1;
    if (p->floor_rps && (!(p->floor_rps[i] >= 0.0f) || !isfinite(p->floor_rps[i]))) return -1;
  }
  return 0;
}

/* Offered load per replica is lambda_i / r, rounded to binary32; the
 * replica runs in the smallest load level that is at least that load.  The
 * paper's load labels are ordinal rungs of an arrival-scale ladder
 * (Section 5, "Workloads and SLOs"); no level large enough -> no option. */
int orc_bucket(const orc_problem *p, int i, int r) {
  float per_replica = p->demand[i] / (float)r;
  for (int b = 0; b < p->n_levels; ++b)
    if (per_replica <= p->levels[b]) return b;
  return -1;
}

/* Satisfaction ratio of r replicas of one configuration, Section 3:
 * x_i <= r * c (Eq. 2), x_i <= lambda_i (Eq. 4), r_i = x_i / lambda_i, and
 * the configuration is usable only if its tail is within the SLO (Eq. 5). */
float orc_fulfillment(const orc_problem *p, int i, float cap, float tail, int r) {
  float capacity = (float)r * cap;
  float ratio = capacity / p->demand[i];
  float f = ratio < 1.0f ? ratio : 1.0f;
  if (!(tail <= p->slo[i])) return 0.0f;
  if (!(f > 0.0f)) return 0.0f; /* a zero ratio is +0 */
  return f;
}

/* Served request rate x_i = min(lambda_i, r * c), binary32. */
static float orc_served(const orc_problem *p, int i, float cap, int r) {
  float capacity = (float)r * cap;
  return capacity < p->demand[i] ? capacity : p->demand[i];
}

/* A critical class's option meets its floor when the configuration is
 * usable (Eq. 5) and serves at least the floor, in req/s. */
static int orc_floor_valid(const orc_problem *p, int i, float cap, float tail, int r) {
  if (!(tail <= p->slo[i])) return 0;
  return orc_served(p, i, cap, r) >= p->floor_rps[i];
}

/* All options of class i: every TP t and replica count r with t*r <= G
 * whose per-replica load falls inside the grid. */
static int orc_class_options(const orc_problem *p, int i, orc_option *opt) {
  int n = 0;
  for (int t = 0; t < p->n_tp; ++t)
    for (int r = 1; p->tp[t] * r <= p->budget; ++r) {
      int b = orc_bucket(p, i, r);
      if (b < 0) continue;
      opt[n].t_idx = t;
      opt[n].r = r;
      opt[n].cost = p->tp[t] * r;
      opt[n].cell = orc_cell(p, i, t, b);
      ++n;
    }
  return n;
}

static int orc_max_options(const orc_problem *p) {
  int n = 0;
  for (int t = 0; t < p->n_tp; ++t) n += p->budget / p->tp[t];
  return n;
}

static void orc_fill_goodput(const orc_problem *p, const float *cap, orc_alloc *a) {
  float goodput = 0.0f;
  int gpus = 0;
  for (int i = 0; i < p->n_classes; ++i) {
    if (a->replicas[i] == 0) continue;
    int t = a->tp_index[i], r = a->replicas[i];
    int cell = orc_cell(p, i, t, orc_bucket(p, i, r));
    goodput += orc_served(p, i, cap[cell], r);
    gpus += p->tp[t] * r;
  }
  a->goodput = goodput;
  a->gpus = gpus;
}

/* ------------------------------------------------------------------ */
/* Solver (i): enumerate every combination and apply the objective.     */
/* ------------------------------------------------------------------ */
int orc_solve_brute(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out) {
  if (orc_check_problem(p)) return -1;
  const int K = p->n_classes;
  const int maxo = orc_max_options(p);
  orc_option *opt = (orc_option *)malloc(sizeof(orc_option) * (size_t)maxo * K);
  float *fval = (float *)malloc(sizeof(float) * (size_t)maxo * K);
  int *fvalid = (int *)malloc(sizeof(int) * (size_t)maxo * K);
  int nopt[ORC_MAX_CLASSES];
  double combos = 1.0;
  for (int i = 0; i < K; ++i) {
    nopt[i] = orc_class_options(p, i, opt + (size_t)i * maxo);
    for (int j = 0; j < nopt[i]; ++j) {
      const orc_option *o = &opt[(size_t)i * maxo + j];
      fval[(size_t)i * maxo + j] = orc_fulfillment(p, i, cap[o->cell], tail[o->cell], o->r);
      fvalid[(size_t)i * maxo + j] =
          orc_is_critical(p, i) ? orc_floor_valid(p, i, cap[o->cell], tail[o->cell], o->r) : 1;
    }
    combos *= (double)(nopt[i] + 1);
  }
  if (combos > 2.0e8) {
    free(opt); free(fval); free(fvalid);
    return -2;
  }
  const int has_crit = orc_has_critical(p);
  int choice[ORC_MAX_CLASSES];

  /* pass 0: can the critical floors be met at all within G?
   * pass 1: best combination under objective level (1) and (2). */
  int floors_feasible = 0;
  int best_found = 0;
  float best_tau = 0.0f;
  int best_gpus = 0;
  int best_tpvec[ORC_MAX_CLASSES];
  int best_choice[ORC_MAX_CLASSES];
  for (int pass = 0; pass < 2; ++pass) {
    if (pass == 0 && !has_crit) continue;
    const int restrict_to_floors = has_crit && floors_feasible;
    for (int i = 0; i < K; ++i) choice[i] = 0;
    for (;;) {
      int gpus = 0, floors_ok = 1;
      float tau = 1.0f;
      int tpvec[ORC_MAX_CLASSES];
      for (int i = 0; i < K; ++i) {
        float f = 0.0f;
        if (choice[i] == 0) {
          tpvec[i] = 0;
          if (orc_is_critical(p, i)) floors_ok = 0;
        } else {
          const orc_option *o = &opt[(size_t)i * maxo + choice[i] - 1];
          gpus += o->cost;
          f = fval[(size_t)i * maxo + choice[i] - 1];
          tpvec[i] = p->tp[o->t_idx];
          if (!fvalid[(size_t)i * maxo + choice[i] - 1]) floors_ok = 0;
        }
        if (f < tau) tau = f;
      }
      if (gpus <= p->budget) {
        if (pass == 0) {
          if (floors_ok) floors_feasible = 1;
        } else if (!restrict_to_floors || floors_ok) {
          int better = 0;
          if (!best_found || tau > best_tau) {
            better = 1;
          } else if (tau == best_tau) {
            if (gpus < best_gpus) {
              better = 1;
            } else if (gpus == best_gpus) {
              for (int i = 0; i < K; ++i) {
                if (tpvec[i] != best_tpvec[i]) {
                  better = tpvec[i] < best_tpvec[i];
                  break;
                }
              }
            }
          }
          if (better) {
            best_found = 1;
            best_tau = tau;
            best_gpus = gpus;
            memcpy(best_tpvec, tpvec, sizeof(int) * K);
            memcpy(best_choice, choice, sizeof(int) * K);
          }
        }
      }
      /* next combination (mixed radix) */
      int i = 0;
      while (i < K) {
        if (++choice[i] <= nopt[i]) break;
        choice[i] = 0;
        ++i;
      }
      if (i == K) break;
    }
  }
  memset(out, 0, sizeof(*out));
  out->tau = best_tau;
  out->floors_met = has_crit ? floors_feasible : 1;
  for (int i = 0; i < K; ++i) {
    if (best_choice[i] == 0) {
      out->tp_index[i] = -1;
      out->replicas[i] = 0;
    } else {
      const orc_option *o = &opt[(size_t)i * maxo + best_choice[i] - 1];
      out->tp_index[i] = o->t_idx;
      out->replicas[i] = o->r;
    }
  }
  orc_fill_goodput(p, cap, out);
  free(opt); free(fval); free(fvalid);
  return 0;
}

/* ------------------------------------------------------------------ */
/* Objective level (1): the floors can be met iff the cheapest floor-   */
/* meeting option of every critical class fits in G together.          */
/* ------------------------------------------------------------------ */
static int orc_floors_feasible(const orc_problem *p, const float *cap, const float *tail,
                               orc_option *opt_scratch) {
  if (!orc_has_critical(p)) return 1;
  long need = 0;
  for (int i = 0; i < p->n_classes; ++i) {
    if (!orc_is_critical(p, i)) continue;
    int n = orc_class_options(p, i, opt_scratch);
    int cheapest = -1;
    for (int j = 0; j < n; ++j) {
      const orc_option *o = &opt_scratch[j];
      if (!orc_floor_valid(p, i, cap[o->cell], tail[o->cell], o->r)) continue;
      if (cheapest < 0 || o->cost < cheapest) cheapest = o->cost;
    }
    if (cheapest < 0) return 0;
    need += cheapest;
  }
  return need <= p->budget;
}

/* ------------------------------------------------------------------ */
/* Solver (ii): (max,min) knapsack over the GPU budget.                 */
/*   B_i[g] = best fulfillment class i reaches with at most g GPUs,     */
/*   D_k[g] = max over a <= g of min(D_{k-1}[g - a], B_k[a]),           */
/*   tau*   = D_K[G];                                                   */
/* then the canonical allocation: each class takes the fewest GPUs that */
/* reach tau* and, among those options, the smallest TP.                */
/* A table entry of -1 means "no allowed choice within this budget".    */
/* ------------------------------------------------------------------ */
int orc_solve_dp(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out) {
  if (orc_check_problem(p)) return -1;
  const int K = p->n_classes, G = p->budget;
  const int maxo = orc_max_options(p);
  orc_option *opt = (orc_option *)malloc(sizeof(orc_option) * (size_t)maxo);
  float *table = (float *)malloc(sizeof(float) * (size_t)(G + 1) * K);
  float *D = (float *)malloc(sizeof(float) * (size_t)(G + 1));
  float *Dn = (float *)malloc(sizeof(float) * (size_t)(G + 1));

  const int has_crit = orc_has_critical(p);
  const int floors_met = orc_floors_feasible(p, cap, tail, opt);
  for (int i = 0; i < K; ++i) {
    float *Bi = table + (size_t)i * (G + 1);
    const int restricted = has_crit && floors_met && orc_is_critical(p, i);
    for (int g = 0; g <= G; ++g) Bi[g] = restricted ? -1.0f : 0.0f;
    int n = orc_class_options(p, i, opt);
    for (int j = 0; j < n; ++j) {
      const orc_option *o = &opt[j];
      if (restricted && !orc_floor_valid(p, i, cap[o->cell], tail[o->cell], o->r)) continue;
      float f = orc_fulfillment(p, i, cap[o->cell], tail[o->cell], o->r);
      if (f > Bi[o->cost]) Bi[o->cost] = f;
    }
    for (int g = 1; g <= G; ++g)
      if (Bi[g - 1] > Bi[g]) Bi[g] = Bi[g - 1];
  }

  float tau;
  if (K == 1) {
    tau = table[G];
  } else {
    memcpy(D, table, sizeof(float) * (size_t)(G + 1));
    for (int k = 1; k < K - 1; ++k) {
      const float *Bk = table + (size_t)k * (G + 1);
      for (int g = 0; g <= G; ++g) {
        float best = -1.0f;
        for (int a = 0; a <= g; ++a) {
          float v = D[g - a] < Bk[a] ? D[g - a] : Bk[a];
          if (v > best) best = v;
        }
        Dn[g] = best;
      }
      memcpy(D, Dn, sizeof(float) * (size_t)(G + 1));
    }
    const float *Bl = table + (size_t)(K - 1) * (G + 1);
    tau = -1.0f;
    for (int a = 0; a <= G; ++a) {
      float v = D[G - a] < Bl[a] ? D[G - a] : Bl[a];
      if (v > tau) tau = v;
    }
  }

  memset(out, 0, sizeof(*out));
  out->tau = tau;
  out->floors_met = floors_met;
  for (int i = 0; i < K; ++i) {
    const float *Bi = table + (size_t)i * (G + 1);
    const int restricted = has_crit && floors_met && orc_is_critical(p, i);
    int m = -1;
    for (int g = 0; g <= G; ++g)
      if (Bi[g] >= tau) { m = g; break; }
    out->tp_index[i] = -1;
    out->replicas[i] = 0;
    if (m <= 0) continue; /* the empty configuration */
    int n = orc_class_options(p, i, opt);
    for (int j = 0; j < n; ++j) { /* options are listed in ascending TP */
      const orc_option *o = &opt[j];
      if (o->cost != m) continue;
      if (restricted && !orc_floor_valid(p, i, cap[o->cell], tail[o->cell], o->r)) continue;
      if (orc_fulfillment(p, i, cap[o->cell], tail[o->cell], o->r) < tau) continue;
      out->tp_index[i] = o->t_idx;
      out->replicas[i] = o->r;
      break;
    }
  }
  orc_fill_goodput(p, cap, out);
  free(opt); free(table); free(D); free(Dn);
  return 0;
}

/* ------------------------------------------------------------------ */
/* Solver (iii): tau* is the largest achievable fulfillment value v for  */
/* which the fewest GPUs each class needs to reach v add up to <= G.     */
/* ------------------------------------------------------------------ */
static int orc_cmp_desc(const void *a, const void *b) {
  float x = *(const float *)a, y = *(const float *)b;
  return (x < y) - (x > y);
}

int orc_solve_threshold(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out) {
  if (orc_check_problem(p)) return -1;
  const int K = p->n_classes;
  const int maxo = orc_max_options(p);
  orc_option *opt = (orc_option *)malloc(sizeof(orc_option) * (size_t)maxo * K);
  float *fval = (float *)malloc(sizeof(float) * (size_t)maxo * K);
  int *allowed = (int *)malloc(sizeof(int) * (size_t)maxo * K);
  float *values = (float *)malloc(sizeof(float) * ((size_t)maxo * K + 1));
  int nopt[ORC_MAX_CLASSES], restricted[ORC_MAX_CLASSES];
  const int has_crit = orc_has_critical(p);

  /* level (1) */
  int floors_met = 1;
  if (has_crit) {
    long need = 0;
    for (int i = 0; i < K && floors_met; ++i) {
      if (!orc_is_critical(p, i)) continue;
      int n = orc_class_options(p, i, opt);
      int cheapest = -1;
      for (int j = 0; j < n; ++j)
        if (orc_floor_valid(p, i, cap[opt[j].cell], tail[opt[j].cell], opt[j].r) &&
            (cheapest < 0 || opt[j].cost < cheapest))
          cheapest = opt[j].cost;
      if (cheapest < 0) floors_met = 0;
      else need += cheapest;
    }
    if (need > p->budget) floors_met = 0;
  }

  int nval = 0;
  values[nval++] = 0.0f;
  for (int i = 0; i < K; ++i) {
    restricted[i] = has_crit && floors_met && orc_is_critical(p, i);
    nopt[i] = orc_class_options(p, i, opt + (size_t)i * maxo);
    for (int j = 0; j < nopt[i]; ++j) {
      const orc_option *o = &opt[(size_t)i * maxo + j];
      float f = orc_fulfillment(p, i, cap[o->cell], tail[o->cell], o->r);
      int ok = restricted[i] ? orc_floor_valid(p, i, cap[o->cell], tail[o->cell], o->r) : 1;
      fval[(size_t)i * maxo + j] = f;
      allowed[(size_t)i * maxo + j] = ok;
      if (ok) values[nval++] = f;
    }
  }
  qsort(values, (size_t)nval, sizeof(float), orc_cmp_desc);

  float tau = -1.0f;
  for (int v = 0; v < nval; ++v) {
    const float target = values[v];
    long need = 0;
    int reachable = 1;
    for (int i = 0; i < K && reachable; ++i) {
      int m = -1;
      if (!restricted[i] && target <= 0.0f) m = 0; /* the empty configuration */
      for (int j = 0; j < nopt[i]; ++j) {
        if (!allowed[(size_t)i * maxo + j] || fval[(size_t)i * maxo + j] < target) continue;
        int c = opt[(size_t)i * maxo + j].cost;
        if (m < 0 || c < m) m = c;
      }
      if (m < 0) reachable = 0;
      else need += m;
    }
    if (reachable && need <= p->budget) {
      tau = target;
      break;
    }
  }
  memset(out, 0, sizeof(*out));
  out->tau = tau;
  out->floors_met = floors_met;
  for (int i = 0; i < K; ++i) out->tp_index[i] = -1;
  free(opt); free(fval); free(allowed); free(values);
  return 0;
}

int orc_solve_batch(const orc_problem *p, const float *cap, const float *tail, int64_t n,
                    orc_alloc *out, int n_threads) {
  if (orc_check_problem(p)) return -1;
  const int64_t N = orc_n_cells(p);
  int err = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
#endif
  for (int64_t j = 0; j < n; ++j) {
    if (orc_solve_dp(p, cap + j * N, tail + j * N, &out[j])) err = -1;
  }
  (void)n_threads;
  return err;
}

/* ------------------------------------------------------------------ */
/* Scores, Section 4.3.                                                 */
/* ------------------------------------------------------------------ */
static double orc_pairwise_rec(const double *x, int64_t n) {
  if (n == 1) return x[0];
  return orc_pairwise_rec(x, n / 2) + orc_pairwise_rec(x + n / 2, n / 2);
}

double orc_pairwise_sum(const double *x, int64_t n) {
  if (n <= 0) return 0.0;
  int64_t p2 = 1;
  while (p2 < n) p2 *= 2;
  double *pad = (double *)calloc((size_t)p2, sizeof(double));
  memcpy(pad, x, sizeof(double) * (size_t)n);
  double s = orc_pairwise_rec(pad, p2);
  free(pad);
  return s;
}

/* Realisations of Section 4.1 for order o: the conservative one pairs
 * every cell's lower capacity bound with its upper tail bound, the
 * optimistic one the upper capacity bound with the lower tail bound. */
static void orc_realisations(int64_t N, int o, const float *cap_lo, const float *cap_hi,
                             const float *tail_lo, const float *tail_hi, float *cap_m,
                             float *tail_m, float *cap_p, float *tail_p) {
  memcpy(cap_m, cap_lo + (size_t)o * N, sizeof(float) * (size_t)N);
  memcpy(tail_m, tail_hi + (size_t)o * N, sizeof(float) * (size_t)N);
  memcpy(cap_p, cap_hi + (size_t)o * N, sizeof(float) * (size_t)N);
  memcpy(tail_p, tail_lo + (size_t)o * N, sizeof(float) * (size_t)N);
}

int orc_score(const orc_problem *p, int32_t n_orders, const float *cap_lo, const float *cap_hi,
              const float *tail_lo, const float *tail_hi, const uint8_t *measured,
              const int32_t *cand, int32_t n_cand, const float *cap_s, const float *tail_s,
              int32_t n_samples, double *score, double *gap_now, int32_t *best, float *tau_dump,
              const uint8_t *tile_mask, int n_threads) {
  if (orc_check_problem(p)) return -1;
  if (n_orders < 0 || n_cand < 0 || n_samples < 1) return -1;
  const int64_t N = orc_n_cells(p);
  const int64_t E = n_cand, S = n_samples;
  for (int e = 0; e < n_cand; ++e)
    if (cand[e] < 0 || cand[e] >= N) return -1;

  float *base_m = (float *)malloc(sizeof(float) * (size_t)(n_orders > 0 ? n_orders : 1));
  float *base_p = (float *)malloc(sizeof(float) * (size_t)(n_orders > 0 ? n_orders : 1));
  int err = 0;

  /* Gamma_t per order: gap between the optimistic and conservative
   * objectives on the current intervals. */
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
#endif
  for (int o = 0; o < n_orders; ++o) {
    float *buf = (float *)malloc(sizeof(float) * (size_t)N * 4);
    orc_alloc am, ap;
    orc_realisations(N, o, cap_lo, cap_hi, tail_lo, tail_hi, buf, buf + N, buf + 2 * N, buf + 3 * N);
    if (orc_solve_dp(p, buf, buf + N, &am) || orc_solve_dp(p, buf + 2 * N, buf + 3 * N, &ap)) err = -1;
    base_m[o] = am.tau;
    base_p[o] = ap.tau;
    gap_now[o] = (double)ap.tau - (double)am.tau;
    free(buf);
  }

  const int64_t tiles = (int64_t)n_orders * E;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
#endif
  for (int64_t tile = 0; tile < tiles; ++tile) {
    if (tile_mask && !tile_mask[tile]) continue;
    const int o = (int)(tile / E);
    const int e = (int)(tile % E);
    const int cell = cand[e];
    if (measured[(size_t)o * N + cell]) {
      /* A revealed cell has nothing left to learn: no scenario is solved,
       * its score is exactly zero and the dump holds the order's base. */
      score[tile] = 0.0;
      if (tau_dump)
        for (int64_t s = 0; s < S; ++s) {
          tau_dump[(tile * S + s) * 2 + 0] = base_m[o];
          tau_dump[(tile * S + s) * 2 + 1] = base_p[o];
        }
      continue;
    }
    float *buf = (float *)malloc(sizeof(float) * (size_t)N * 4);
    double *gam = (double *)malloc(sizeof(double) * (size_t)S);
    float *cap_m = buf, *tail_m = buf + N, *cap_p = buf + 2 * N, *tail_p = buf + 3 * N;
    orc_realisations(N, o, cap_lo, cap_hi, tail_lo, tail_hi, cap_m, tail_m, cap_p, tail_p);
    for (int64_t s = 0; s < S; ++s) {
      /* Scenario (o, e, s): cell e takes the sampled outcome in both
       * realisations; Gamma_{t+1} is the gap that would remain. */
      const float cs = cap_s[tile * S + s], ts = tail_s[tile * S + s];
      cap_m[cell] = cs; tail_m[cell] = ts;
      cap_p[cell] = cs; tail_p[cell] = ts;
      orc_alloc am, ap;
      if (orc_solve_dp(p, cap_m, tail_m, &am) || orc_solve_dp(p, cap_p, tail_p, &ap)) err = -1;
      gam[s] = (double)ap.tau - (double)am.tau;
      if (tau_dump) {
        tau_dump[(tile * S + s) * 2 + 0] = am.tau;
        tau_dump[(tile * S + s) * 2 + 1] = ap.tau;
      }
    }
    score[tile] = gap_now[o] - orc_pairwise_sum(gam, S) / (double)S;
    free(buf);
    free(gam);
  }

  /* Reveal the candidate with the largest expected gap reduction; the
   * expected profiling GPU-seconds (cell duration x TP) break ties, then
   * the smaller cell index, then the earlier candidate. */
  for (int o = 0; o < n_orders; ++o) {
    int b = -1;
    for (int e = 0; e < n_cand; ++e) {
      const int cell = cand[e];
      if (measured[(size_t)o * N + cell]) continue;
      if (b < 0) { b = e; continue; }
      const double se = score[(size_t)o * E + e], sb = score[(size_t)o * E + b];
      const int te = p->tp[(cell / p->n_levels) % p->n_tp];
      const int tb = p->tp[(cand[b] / p->n_levels) % p->n_tp];
      if (se > sb || (se == sb && (te < tb || (te == tb && cell < cand[b])))) b = e;
    }
    best[o] = b;
  }
  free(base_m);
  free(base_p);
  return err;
}

/* ------------------------------------------------------------------ */
/* Certificate, Section 4.2 and Algorithm 1.                            */
/* ------------------------------------------------------------------ */
int orc_certify(const orc_problem *p, int32_t n_orders, const float *cap_lo, const float *cap_hi,
                const float *tail_lo, const float *tail_hi, const uint8_t *measured, float eps,
                int32_t *state, orc_alloc *cons, orc_alloc *opt, double *gap) {
  if (orc_check_problem(p)) return -1;
  const int64_t N = orc_n_cells(p);
  const int has_crit = orc_has_critical(p);
  float *buf = (float *)malloc(sizeof(float) * (size_t)N * 4);
  for (int o = 0; o < n_orders; ++o) {
    orc_realisations(N, o, cap_lo, cap_hi, tail_lo, tail_hi, buf, buf + N, buf + 2 * N, buf + 3 * N);
    orc_solve_dp(p, buf, buf + N, &cons[o]);
    orc_solve_dp(p, buf + 2 * N, buf + 3 * N, &opt[o]);
    gap[o] = (double)opt[o].tau - (double)cons[o].tau;
    if (has_crit && !opt[o].floors_met) {
      /* even the optimistic allocation cannot meet a critical floor */
      state[o] = ORC_CERTIFIED_INFEASIBLE;
      continue;
    }
    int ok = cons[o].floors_met;
    /* every configuration the conservative allocation commits to must have
     * a measured (known) tail upper bound that is within the SLO */
    for (int i = 0; i < p->n_classes && ok; ++i) {
      if (cons[o].replicas[i] == 0) continue;
      const int r = cons[o].replicas[i];
      const int cell = orc_cell(p, i, cons[o].tp_index[i], orc_bucket(p, i, r));
      if (!measured[(size_t)o * N + cell]) ok = 0;
      else if (!(tail_hi[(size_t)o * N + cell] <= p->slo[i])) ok = 0;
    }
    if (ok && gap[o] <= (double)eps) state[o] = ORC_CERTIFIED_FEASIBLE;
    else state[o] = ORC_UNDECIDED;
  }
  free(buf);
  return 0;
}

/* ------------------------------------------------------------------ */
/* The whole lexicographic objective, levels (1)-(4).                   */
/* ------------------------------------------------------------------ */

/* Served goodput of an option: failed requests are not goodput, so a
 * configuration whose tail breaks the SLO serves 0. */
static float orc_goodput_served(const orc_problem *p, int i, float cap, float tail, int r) {
  if (!(tail <= p->slo[i])) return 0.0f;
  return orc_served(p, i, cap, r);
}

/* Key of the residual tie-break: (TP degree, replicas) of class i, empty =
 * (0, 0). */
static int orc_lex_cmp(const orc_problem *p, const int *tpi_a, const int *r_a, const int *tpi_b,
                       const int *r_b) {
  for (int i = 0; i < p->n_classes; ++i) {
    const int ta = tpi_a[i] < 0 ? 0 : p->tp[tpi_a[i]], tb = tpi_b[i] < 0 ? 0 : p->tp[tpi_b[i]];
    if (ta != tb) return ta < tb ? -1 : 1;
    if (r_a[i] != r_b[i]) return r_a[i] < r_b[i] ? -1 : 1;
  }
  return 0;
}

int orc_solve_lex_brute(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out,
                        double *goodput64) {
  if (orc_check_problem(p)) return -1;
  const int K = p->n_classes;
  const int maxo = orc_max_options(p);
  orc_option *opt = (orc_option *)malloc(sizeof(orc_option) * (size_t)maxo * K);
  int nopt[ORC_MAX_CLASSES];
  double combos = 1.0;
  for (int i = 0; i < K; ++i) {
    nopt[i] = orc_class_options(p, i, opt + (size_t)i * maxo);
    combos *= (double)(nopt[i] + 1);
  }
  if (combos > 2.0e8) {
    free(opt);
    return -2;
  }
  const int has_crit = orc_has_critical(p);
  int choice[ORC_MAX_CLASSES];
  int floors_feasible = 0, best_found = 0, best_gpus = 0;
  float best_tau = 0.0f;
  double best_gp = 0.0;
  int best_tpi[ORC_MAX_CLASSES], best_r[ORC_MAX_CLASSES];
  for (int pass = 0; pass < 2; ++pass) {
    if (pass == 0 && !has_crit) continue;
    const int restrict_to_floors = has_crit && floors_feasible;
    for (int i = 0; i < K; ++i) choice[i] = 0;
    for (;;) {
      int gpus = 0, floors_ok = 1;
      float tau = 1.0f;
      int tpi[ORC_MAX_CLASSES], rr[ORC_MAX_CLASSES];
      float served[ORC_MAX_CLASSES];
      for (int i = 0; i < K; ++i) {
        float f = 0.0f;
        served[i] = 0.0f;
        tpi[i] = -1;
        rr[i] = 0;
        if (choice[i] == 0) {
          if (orc_is_critical(p, i)) floors_ok = 0;
        } else {
          const orc_option *o = &opt[(size_t)i * maxo + choice[i] - 1];
          const float c = cap[o->cell], l = tail[o->cell];
          gpus += o->cost;
          f = orc_fulfillment(p, i, c, l, o->r);
          served[i] = orc_goodput_served(p, i, c, l, o->r);
          tpi[i] = o->t_idx;
          rr[i] = o->r;
          if (orc_is_critical(p, i) && !orc_floor_valid(p, i, c, l, o->r)) floors_ok = 0;
        }
        if (f < tau) tau = f;
      }
      if (gpus <= p->budget) {
        if (pass == 0) {
          if (floors_ok) floors_feasible = 1;
        } else if (!restrict_to_floors || floors_ok) {
          double gp = 0.0;
          for (int i = K - 1; i >= 0; --i) gp = (double)served[i] + gp;
          int better = 0;
          if (!best_found) better = 1;
          else if (tau != best_tau) better = tau > best_tau;
          else if (gp != best_gp) better = gp > best_gp;
          else if (gpus != best_gpus) better = gpus < best_gpus;
          else better = orc_lex_cmp(p, tpi, rr, best_tpi, best_r) < 0;
          if (better) {
            best_found = 1;
            best_tau = tau;
            best_gp = gp;
            best_gpus = gpus;
            memcpy(best_tpi, tpi, sizeof(int) * K);
            memcpy(best_r, rr, sizeof(int) * K);
          }
        }
      }
      int i = 0;
      while (i < K) {
        if (++choice[i] <= nopt[i]) break;
        choice[i] = 0;
        ++i;
      }
      if (i == K) break;
    }
  }
  memset(out, 0, sizeof(*out));
  out->tau = best_tau;
  out->floors_met = has_crit ? floors_feasible : 1;
  for (int i = 0; i < K; ++i) {
    out->tp_index[i] = best_tpi[i];
    out->replicas[i] = best_r[i];
  }
  orc_fill_goodput(p, cap, out);
  if (goodput64) *goodput64 = best_gp;
  free(opt);
  return 0;
}

/* Levels (3)-(4) as a knapsack over the budget, classes taken from the
 * last to the first:
 *   V_K[g] = (0, 0 GPUs) for every g;
 *   V_k[g] = best over the allowed options o of class k with cost <= g of
 *            (served_o + V_{k+1}[g - cost].goodput, cost + V_{k+1}[g - cost].gpus),
 * best = larger goodput, then fewer GPUs.  Allowed: ratio >= tau* (level 2),
 * floor-meeting for a critical class when the floors are enforced (level
 * 1), and the empty option only for an unrestricted class when tau* = 0.
 * The allocation is then read in class order: class k takes the first
 * allowed option, in (TP, replicas) order with empty first, that keeps the
 * optimum of V_k at the remaining budget. */
int orc_solve_lex(const orc_problem *p, const float *cap, const float *tail, orc_alloc *out,
                  double *goodput64) {
  if (orc_check_problem(p)) return -1;
  orc_alloc base;
  int err = orc_solve_dp(p, cap, tail, &base);
  if (err) return err;
  const int K = p->n_classes, G = p->budget;
  const float tau = base.tau;
  const int has_crit = orc_has_critical(p);
  const int maxo = orc_max_options(p);
  orc_option *opt = (orc_option *)malloc(sizeof(orc_option) * (size_t)maxo * K);
  int *allowed = (int *)malloc(sizeof(int) * (size_t)maxo * K);
  float *served = (float *)malloc(sizeof(float) * (size_t)maxo * K);
  int nopt[ORC_MAX_CLASSES], empty_ok[ORC_MAX_CLASSES];
  for (int i = 0; i < K; ++i) {
    const int restricted = has_crit && base.floors_met && orc_is_critical(p, i);
    empty_ok[i] = !restricted && tau <= 0.0f;
    nopt[i] = orc_class_options(p, i, opt + (size_t)i * maxo);
    for (int j = 0; j < nopt[i]; ++j) {
      const orc_option *o = &opt[(size_t)i * maxo + j];
      const float c = cap[o->cell], l = tail[o->cell];
      int ok = orc_fulfillment(p, i, c, l, o->r) >= tau;
      if (restricted && !orc_floor_valid(p, i, c, l, o->r)) ok = 0;
      allowed[(size_t)i * maxo + j] = ok;
      served[(size_t)i * maxo + j] = orc_goodput_served(p, i, c, l, o->r);
    }
  }
  /* layer k at offset k * (G + 1); gpus < 0 marks "no allowed completion" */
  double *vgp = (double *)malloc(sizeof(double) * (size_t)(K + 1) * (G + 1));
  int *vgpus = (int *)malloc(sizeof(int) * (size_t)(K + 1) * (G + 1));
  for (int g = 0; g <= G; ++g) {
    vgp[(size_t)K * (G + 1) + g] = 0.0;
    vgpus[(size_t)K * (G + 1) + g] = 0;
  }
  for (int k = K - 1; k >= 0; --k) {
    const double *ngp = vgp + (size_t)(k + 1) * (G + 1);
    const int *ngpus = vgpus + (size_t)(k + 1) * (G + 1);
    for (int g = 0; g <= G; ++g) {
      double bgp = 0.0;
      int bgpus = -1;
      if (empty_ok[k] && ngpus[g] >= 0) {
        bgp = ngp[g];
        bgpus = ngpus[g];
      }
      for (int j = 0; j < nopt[k]; ++j) {
        const orc_option *o = &opt[(size_t)k * maxo + j];
        if (!allowed[(size_t)k * maxo + j] || o->cost > g || ngpus[g - o->cost] < 0) continue;
        const double cgp = (double)served[(size_t)k * maxo + j] + ngp[g - o->cost];
        const int cgpus = o->cost + ngpus[g - o->cost];
        if (bgpus < 0 || cgp > bgp || (cgp == bgp && cgpus < bgpus)) {
          bgp = cgp;
          bgpus = cgpus;
        }
      }
      vgp[(size_t)k * (G + 1) + g] = bgp;
      vgpus[(size_t)k * (G + 1) + g] = bgpus;
    }
  }
  memset(out, 0, sizeof(*out));
  out->tau = tau;
  out->floors_met = base.floors_met;
  int rem = G;
  for (int k = 0; k < K; ++k) {
    const double want_gp = vgp[(size_t)k * (G + 1) + rem];
    const int want_gpus = vgpus[(size_t)k * (G + 1) + rem];
    const double *ngp = vgp + (size_t)(k + 1) * (G + 1);
    const int *ngpus = vgpus + (size_t)(k + 1) * (G + 1);
    out->tp_index[k] = -1;
    out->replicas[k] = 0;
    if (empty_ok[k] && ngpus[rem] >= 0 && ngp[rem] == want_gp && ngpus[rem] == want_gpus) continue;
    /* options are listed by TP index, then replicas: (TP degree, r) order */
    for (int j = 0; j < nopt[k]; ++j) {
      const orc_option *o = &opt[(size_t)k * maxo + j];
      if (!allowed[(size_t)k * maxo + j] || o->cost > rem || ngpus[rem - o->cost] < 0) continue;
      if ((double)served[(size_t)k * maxo + j] + ngp[rem - o->cost] != want_gp) continue;
      if (o->cost + ngpus[rem - o->cost] != want_gpus) continue;
      out->tp_index[k] = o->t_idx;
      out->replicas[k] = o->r;
      rem -= o->cost;
      break;
    }
  }
  orc_fill_goodput(p, cap, out);
  if (goodput64) *goodput64 = vgp[G];
  free(opt); free(allowed); free(served); free(vgp); free(vgpus);
  return 0;
}

int orc_certify_lex(const orc_problem *p, int32_t n_orders, const float *cap_lo, const float *cap_hi,
                    const float *tail_lo, const float *tail_hi, const uint8_t *measured, float eps,
                    int32_t *state, orc_alloc *cons, orc_alloc *opt, double *gap_mm, double *gap_gp) {
  if (orc_check_problem(p)) return -1;
  const int64_t N = orc_n_cells(p);
  const int has_crit = orc_has_critical(p);
  float *buf = (float *)malloc(sizeof(float) * (size_t)N * 4);
  for (int o = 0; o < n_orders; ++o) {
    double gp_m = 0.0, gp_p = 0.0;
    orc_realisations(N, o, cap_lo, cap_hi, tail_lo, tail_hi, buf, buf + N, buf + 2 * N, buf + 3 * N);
    orc_solve_lex(p, buf, buf + N, &cons[o], &gp_m);
    orc_solve_lex(p, buf + 2 * N, buf + 3 * N, &opt[o], &gp_p);
    gap_mm[o] = (double)opt[o].tau - (double)cons[o].tau;
    const double top = gp_p > gp_m ? gp_p : gp_m;
    gap_gp[o] = top > 0.0 ? fabs(gp_p - gp_m) / top : 0.0;
    if (has_crit && !opt[o].floors_met) {
      state[o] = ORC_CERTIFIED_INFEASIBLE;
      continue;
    }
    int ok = cons[o].floors_met;
    for (int i = 0; i < p->n_classes && ok; ++i) {
      if (cons[o].replicas[i] == 0) continue;
      const int r = cons[o].replicas[i];
      const int cell = orc_cell(p, i, cons[o].tp_index[i], orc_bucket(p, i, r));
      if (!measured[(size_t)o * N + cell]) ok = 0;
      else if (!(tail_hi[(size_t)o * N + cell] <= p->slo[i])) ok = 0;
    }
    if (ok && gap_mm[o] <= (double)eps && gap_gp[o] <= (double)eps) state[o] = ORC_CERTIFIED_FEASIBLE;
    else state[o] = ORC_UNDECIDED;
  }
  free(buf);
  return 0;
}

/* Stage-wise gap of one pair of allocations under the whole objective:
 * max-min stage tau+ - tau-, goodput stage |gp+ - gp-| / max(gp+, gp-). */
static void orc_stage_gaps(const orc_alloc *am, const orc_alloc *ap, double gm, double gp, double *mm,
                           double *gg) {
  *mm = (double)ap->tau - (double)am->tau;
  const double top = gp > gm ? gp : gm;
  *gg = top > 0.0 ? fabs(gp - gm) / top : 0.0;
}

int orc_score_lex(const orc_problem *p, int32_t n_orders, const float *cap_lo, const float *cap_hi,
                  const float *tail_lo, const float *tail_hi, const uint8_t *measured, const int32_t *cand,
                  int32_t n_cand, const float *cap_s, const float *tail_s, int32_t n_samples, double *score_mm,
                  double *score_gp, double *gap_mm, double *gap_gp, int32_t *best, const uint8_t *tile_mask,
                  int n_threads) {
  if (orc_check_problem(p)) return -1;
  if (n_orders < 0 || n_cand < 0 || n_samples < 1) return -1;
  const int64_t N = orc_n_cells(p);
  const int64_t E = n_cand, S = n_samples;
  for (int e = 0; e < n_cand; ++e)
    if (cand[e] < 0 || cand[e] >= N) return -1;
  int err = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
#endif
  for (int o = 0; o < n_orders; ++o) {
    float *buf = (float *)malloc(sizeof(float) * (size_t)N * 4);
    orc_alloc am, ap;
    double gm = 0.0, gp = 0.0;
    orc_realisations(N, o, cap_lo, cap_hi, tail_lo, tail_hi, buf, buf + N, buf + 2 * N, buf + 3 * N);
    if (orc_solve_lex(p, buf, buf + N, &am, &gm) || orc_solve_lex(p, buf + 2 * N, buf + 3 * N, &ap, &gp)) err = -1;
    orc_stage_gaps(&am, &ap, gm, gp, &gap_mm[o], &gap_gp[o]);
    free(buf);
  }
  const int64_t tiles = (int64_t)n_orders * E;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads > 0 ? n_threads : 1)
#endif
  for (int64_t tile = 0; tile < tiles; ++tile) {
    if (tile_mask && !tile_mask[tile]) continue;
    const int o = (int)(tile / E);
    const int e = (int)(tile % E);
    const int cell = cand[e];
    if (measured[(size_t)o * N + cell]) {
      score_mm[tile] = 0.0;
      score_gp[tile] = 0.0;
      continue;
    }
    float *buf = (float *)malloc(sizeof(float) * (size_t)N * 4);
    double *gmm = (double *)malloc(sizeof(double) * (size_t)S);
    double *ggp = (double *)malloc(sizeof(double) * (size_t)S);
    float *cap_m = buf, *tail_m = buf + N, *cap_p = buf + 2 * N, *tail_p = buf + 3 * N;
    orc_realisations(N, o, cap_lo, cap_hi, tail_lo, tail_hi, cap_m, tail_m, cap_p, tail_p);
    for (int64_t s = 0; s < S; ++s) {
      const float cs = cap_s[tile * S + s], ts = tail_s[tile * S + s];
      cap_m[cell] = cs; tail_m[cell] = ts;
      cap_p[cell] = cs; tail_p[cell] = ts;
      orc_alloc am, ap;
      double gm = 0.0, gp = 0.0;
      if (orc_solve_lex(p, cap_m, tail_m, &am, &gm) || orc_solve_lex(p, cap_p, tail_p, &ap, &gp)) err = -1;
      orc_stage_gaps(&am, &ap, gm, gp, &gmm[s], &ggp[s]);
    }
    score_mm[tile] = gap_mm[o] - orc_pairwise_sum(gmm, S) / (double)S;
    score_gp[tile] = gap_gp[o] - orc_pairwise_sum(ggp, S) / (double)S;
    free(buf);
    free(gmm);
    free(ggp);
  }
  /* the larger expected max-min reduction, then the larger expected
   * goodput-stage reduction, then the cheaper cell, the smaller cell, the
   * earlier candidate */
  for (int o = 0; o < n_orders; ++o) {
    int b = -1;
    for (int e = 0; e < n_cand; ++e) {
      const int cell = cand[e];
      if (measured[(size_t)o * N + cell]) continue;
      if (b < 0) { b = e; continue; }
      const double me = score_mm[(size_t)o * E + e], mb = score_mm[(size_t)o * E + b];
      const double ge = score_gp[(size_t)o * E + e], gb = score_gp[(size_t)o * E + b];
      const int te = p->tp[(cell / p->n_levels) % p->n_tp];
      const int tb = p->tp[(cand[b] / p->n_levels) % p->n_tp];
      int better;
      if (me != mb) better = me > mb;
      else if (ge != gb) better = ge > gb;
      else if (te != tb) better = te < tb;
      else better = cell < cand[b];
      if (better) b = e;
    }
    best[o] = b;
  }
  return err;
}
