// fs_kernels.hip -- gfx950 kernels of libfleetsieve.
//
// The allocation (FleetSieve, Section 3, Eq. 1-5): class i picks one
// configuration, t GPUs per replica and r replicas (t * r GPUs), or nothing;
// its satisfaction ratio is min(1, fl32(fl32(r * c) / lambda_i)) when the
// configuration's tail is within the SLO (Eq. 5), else 0; the total GPUs are
// at most G (Eq. 3); the objective maximises the minimum ratio over classes
// after enforcing critical floors whenever they can be met.  Its value is
// tau* = D_K[G] of the (max,min) knapsack
//   B_i[g] = best ratio of class i with at most g GPUs,
//   D_1 = B_1,  D_k[g] = max_{a <= g} min(D_{k-1}[g - a], B_k[a]).
// Tie-breaks (fewer GPUs, then the lexicographically smaller TP vector) are
// resolved after tau* is known: each class takes the fewest GPUs reaching
// tau* and, among those options, the smallest TP.
//
// Two kernel families:
//  * wave-per-scenario (any problem): one wavefront owns a scenario; per-class
//    tables live in LDS; options are spread over lanes and merged with LDS
//    atomic max; prefix maxima use a wave scan; the DP spreads budgets over
//    lanes and reduces with cross-lane max.
//  * lane-per-scenario (no floors, TP set {1,2,4,8}, G in {16,32,64}): one
//    lane owns a scenario; the 64 lanes of a wavefront are 64 samples of the
//    same (order, candidate), so the order's option values are wave-uniform
//    scalar loads and only the candidate's own cell differs per lane.  All
//    tables are register-resident and the DP is fully unrolled.
//
// Fulfillment values are compared as int32 bit patterns: for binary32 values
// >= +0 the integer order is the float order, -1 marks "no allowed choice"
// (critical floors) and a -0 ratio (from a -0 capacity) sorts below every
// usable value, which is how a zero ratio behaves in the max.
#include "fs_internal.h"

#include <limits.h>

namespace fs {

namespace {

// ---------------------------------------------------------------------------
// Scalar helpers shared by both kernel families.
// ---------------------------------------------------------------------------

// Ratio of r replicas of a cell (cap, tail) for a class with SLO `slo` and
// demand reciprocal `rcp`, as int32 bits (0 when the tail breaks the SLO).
__device__ __forceinline__ int ratio_bits(float cap, float tail, int r, float slo, double rcp) {
  const float capacity = (float)r * cap;
  const float q = (float)((double)capacity * rcp);
  const float f = fminf(q, 1.0f);
  return (tail <= slo) ? __float_as_int(f) : 0;
}

__device__ __forceinline__ float served_rps(float cap, int r, float demand) {
  const float capacity = (float)r * cap;
  return capacity < demand ? capacity : demand;
}

__device__ __forceinline__ bool floor_ok(float cap, float tail, int r, float slo, float demand,
                                         float floor_rps) {
  return (tail <= slo) && served_rps(cap, r, demand) >= floor_rps;
}

__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, __shfl_xor(v, off, kWave));
  return v;
}

__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = min(v, __shfl_xor(v, off, kWave));
  return v;
}

// Inclusive prefix maximum across the 64 lanes.
__device__ __forceinline__ int wave_scan_max(int v, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(v, off, kWave);
    if (lane >= off) v = max(v, t);
  }
  return v;
}

// Inclusive prefix sum across the 64 lanes by DPP: shifts by 1, 2, 4, 8
// within each row of 16 lanes (lanes with no source add 0), then the last
// lane of row 0 is added to row 1 and of row 2 to row 3 (row_bcast:15), and
// the last lane of row 1 (the total of rows 0-1) to rows 2 and 3
// (row_bcast:31).
__device__ __forceinline__ int wave_scan_add(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// Maximum / minimum over the 64 lanes: DPP permutations within each row of
// 16 lanes (quad xor 1, quad xor 2, half-row mirror, row mirror), then the
// four row results by readlane.  Wave-uniform result; every lane must be
// active.
__device__ __forceinline__ int wave_max_dpp(int v) {
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, true));
  return max(max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

__device__ __forceinline__ int wave_min_dpp(int v) {
  v = min(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));
  v = min(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));
  v = min(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, true));
  v = min(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, true));
  return min(min(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             min(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

// Sum over the 64 lanes (wave-uniform result; every lane must be active).
__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Inclusive prefix maximum of nonnegative values across the 64 lanes: DPP
// shifts by 1, 2, 4, 8 within each row (a lane with no source takes 0), then
// every row takes the totals of the rows before it (by readlane).
__device__ __forceinline__ int wave_scan_max_nonneg(int v, int lane) {
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false));  // row_shr:1
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false));  // row_shr:2
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false));  // row_shr:4
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false));  // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31);
  const int r2 = __builtin_amdgcn_readlane(v, 47);
  const int row = lane >> 4;
  const int before = row == 0 ? 0 : row == 1 ? r0 : row == 2 ? max(r0, r1) : max(max(r0, r1), r2);
  return max(v, before);
}

// Inclusive prefix sum across the 64 lanes: the same DPP shifts within rows,
// then the totals of the rows before.
__device__ __forceinline__ int wave_scan_add_rows(int v, int lane) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);
  const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31);
  const int r2 = __builtin_amdgcn_readlane(v, 47);
  const int row = lane >> 4;
  return v + (row == 0 ? 0 : row == 1 ? r0 : row == 2 ? r0 + r1 : r0 + r1 + r2);
}

// One DPP lane permutation of a binary64 value (both halves moved alike).
template <int kCtrl>
__device__ __forceinline__ double dpp_f64(double v) {
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), kCtrl, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), kCtrl, 0xF, 0xF, true);
  return __hiloint2double(hi, lo);
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
  return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(v), l),
                          __builtin_amdgcn_readlane(__double2loint(v), l));
}

// Pairwise sum over the 64 lanes, as the balanced binary tree over lane
// order: after each step every lane holds the sum of its aligned block of
// 2, 4, 8, 16 lanes (the partner block's value comes by a DPP permutation:
// quad xor 1, quad xor 2, half-row mirror, row mirror; every lane of a block
// holds the same sum, and a + b = b + a exactly), then the four row sums are
// combined as (r0 + r1) + (r2 + r3).  The result is the same in every lane.
__device__ __forceinline__ double wave_pairwise_sum(double v) {
  v = v + dpp_f64<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v = v + dpp_f64<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v = v + dpp_f64<0x141>(v);  // row_half_mirror
  v = v + dpp_f64<0x140>(v);  // row_mirror
  return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

// Orders LDS accesses of one wavefront (its lanes' writes before their
// reads); LDS executes one wavefront's instructions in issue order.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int cell_of(const DevProblem &P, int k, int ti, int b) {
  return (k * P.NT + ti) * P.B + b;
}

// ---------------------------------------------------------------------------
// Set-up: load level of every (class, replica count), and candidate info.
// ---------------------------------------------------------------------------
// Load level of r replicas of class k: the offered load per replica is
// lambda_k / r in binary32, and the replica runs in the smallest level that
// is at least that load; -1 when no level is large enough.  level_from takes
// the per-replica load; its loop runs over the largest level count, so the
// levels (kernel arguments) come in a few wide scalar loads rather than one
// per compare.
__device__ __forceinline__ int level_from(const DevProblem &P, float per_replica) {
  int b = -1;
#pragma unroll
  for (int j = kMaxLevels - 1; j >= 0; --j) b = (j < P.B && per_replica <= P.levels[j]) ? j : b;
  return b;
}

__device__ __forceinline__ int level_of(const DevProblem &P, int k, int r) {
  return level_from(P, P.demand[k] / (float)r);
}

// Number of load levels below a per-replica load: the index of the smallest
// level that holds it, B when none does.  The loop runs over the largest
// level count, so the level values (kernel arguments) are fetched by a few
// wide scalar loads ahead of the compares instead of one load per level.
__device__ __forceinline__ int levels_below(const DevProblem &P, float per_replica) {
  int b = 0;
#pragma unroll
  for (int j = 0; j < kMaxLevels; ++j) b += (j < P.B && P.levels[j] < per_replica) ? 1 : 0;
  return b;
}

// Copies n bytes to LDS with all of a thread's loads (up to 8) issued before
// its first LDS write, so their latencies overlap.
__device__ __forceinline__ void stage_u8(uint8_t *__restrict__ dst, const uint8_t *__restrict__ src, int n,
                                         int tid, int nth) {
  for (int x0 = tid; x0 < n; x0 += 8 * nth) {
    uint8_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = x0 + u * nth < n ? src[x0 + u * nth] : 0;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (x0 + u * nth < n) dst[x0 + u * nth] = v[u];
  }
}

// Bucket map entry idx = k (G + 1) + r: the load level of r replicas of
// class k (-1 for r = 0).
__device__ __forceinline__ void setup_bucket_at(const DevProblem &P, int8_t *__restrict__ bmap, int idx) {
  const int n = P.K * (P.G + 1);
  if (idx >= n) return;
  const int k = idx / (P.G + 1), r = idx % (P.G + 1);
  bmap[idx] = (int8_t)(r >= 1 ? level_of(P, k, r) : -1);
}

// Z[g] = max_{a <= g} min(X[g - a], Y[a]) for nondecreasing X and Y.  The
// inner minimum follows Y while Y[a] < X[g - a] and X afterwards, so it rises
// and then falls in a; with a* the first a where Y[a] >= X[g - a] (a
// monotone predicate, found by bisection) the maximum is
// max(Y[a* - 1], X[g - a*]).  `top` is a power of two with 2 * top > g + 1.
__device__ __forceinline__ int conv_mono(const int *X, const int *Y, int g, int top) {
  int pos = 0;
  for (int step = top; step > 0; step >>= 1) {
    const int a = min(pos + step - 1, g);
    const bool below = Y[a] < X[g - a];
    pos += (pos + step - 1 <= g && below) ? step : 0;
  }
  const int left = Y[max(pos - 1, 0)];
  const int right = X[g - min(pos, g)];
  return max(pos >= 1 ? left : INT_MIN, pos <= g ? right : INT_MIN);
}

// Entries of X among the first d entries of the ascending merge of X and Y
// (n entries each, X first among equal values): a bisection over the split.
__device__ __forceinline__ int merge_split(const int *X, const int *Y, int n, int d) {
  int lo = max(0, d - n), hi = min(d, n);
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (X[mid] <= Y[d - 1 - mid]) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Folds options into their cells' maxima and replica ranges.  Lanes holding
// consecutive options of one TP degree fall on few cells (the load level
// falls as r grows), in runs of lanes; the first lane of each run folds the
// run's largest value and replica range in with one LDS atomic each, where
// one per lane would queue up on the same bank.  key: the cell within the
// class, -1 for a lane with no option.  Every lane of the wavefront calls
// it (the shuffles read every lane); r grows along a run.
__device__ __forceinline__ void fold_cell_runs(int key, int w, int r, int *mc, int *crlo, int *crhi) {
  const int lane = threadIdx.x & (kWave - 1);
  int wmax = w, rmax = r;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int k2 = __shfl_down(key, d, kWave);
    const int w2 = __shfl_down(wmax, d, kWave);
    const int r2 = __shfl_down(rmax, d, kWave);
    const bool in = lane + d < kWave && k2 == key;
    wmax = in ? max(wmax, w2) : wmax;
    rmax = in ? max(rmax, r2) : rmax;
  }
  const int kprev = __shfl_up(key, 1, kWave);
  if (key >= 0 && (lane == 0 || kprev != key)) {
    atomicMax(&mc[key], wmax);
    atomicMin(&crlo[key], r);
    atomicMax(&crhi[key], rmax);
  }
}

// ---------------------------------------------------------------------------
// Wave-per-scenario solver.
// ---------------------------------------------------------------------------

// A point realisation: base cell arrays with at most one cell replaced.
struct Realisation {
  const float *cap;
  const float *tail;
  int ocell;
  float ocap, otail;
  __device__ __forceinline__ float c(int cell) const { return cell == ocell ? ocap : cap[cell]; }
  __device__ __forceinline__ float l(int cell) const { return cell == ocell ? otail : tail[cell]; }
};

struct WaveAlloc {  // optional per-class allocation (LDS), filled on request
  int *tp_index;    // [K] -1 = none
  int *replicas;    // [K]
};

// Solves one realisation with the whole wavefront.  lds must hold
// 3 * (G + 1) ints.  Returns tau* as int32 bits; *floors_met receives
// objective level (1)'s outcome.  When alloc is non-null, the canonical
// allocation is written to it and *goodput (lane 0) receives the served total.
__device__ int wave_solve(const DevProblem &P, const int8_t *__restrict__ bmap,
                          const Realisation &R, int *lds, int *floors_met_out,
                          const WaveAlloc *alloc, float *goodput) {
  const int lane = threadIdx.x & (kWave - 1);
  const int K = P.K, G = P.G;

  // Objective level (1): can every critical floor be met within G?
  int floors_met = 1;
  if (P.has_floor) {
    int need = 0;
    bool ok = true;
    for (int k = 0; k < K && ok; ++k) {
      if (!(P.floor_rps[k] > 0.0f)) continue;
      int cheapest = INT_MAX;
      for (int ti = 0; ti < P.NT; ++ti) {
        const int t = P.tp[ti];
        for (int r = 1 + lane; t * r <= G; r += kWave) {
          const int b = bmap[k * (G + 1) + r];
          if (b < 0) continue;
          const int cell = cell_of(P, k, ti, b);
          if (floor_ok(R.c(cell), R.l(cell), r, P.slo[k], P.demand[k], P.floor_rps[k]))
            cheapest = min(cheapest, t * r);
        }
      }
      cheapest = wave_min(cheapest);
      if (cheapest == INT_MAX) ok = false;
      else need += cheapest;
    }
    floors_met = (ok && need <= G) ? 1 : 0;
  }
  *floors_met_out = floors_met;

  int *D = lds, *T = lds + (G + 1), *Dn = lds + 2 * (G + 1);
  int top = 1;
  while (2 * top <= G + 1) top <<= 1;  // 2 top > G + 1 >= g + 1: the crossing search covers [0, g]
  int tau = 0;
  for (int k = 0; k < K; ++k) {
    const bool restricted = P.has_floor && floors_met && (P.floor_rps[k] > 0.0f);
    const int init = restricted ? -1 : 0;
    for (int g = lane; g <= G; g += kWave) T[g] = init;
    __syncthreads();
    for (int ti = 0; ti < P.NT; ++ti) {
      const int t = P.tp[ti];
      for (int r = 1 + lane; t * r <= G; r += kWave) {
        const int b = bmap[k * (G + 1) + r];
        if (b < 0) continue;
        const int cell = cell_of(P, k, ti, b);
        const float c = R.c(cell), l = R.l(cell);
        if (restricted && !floor_ok(c, l, r, P.slo[k], P.demand[k], P.floor_rps[k])) continue;
        atomicMax(&T[t * r], ratio_bits(c, l, r, P.slo[k], P.rcp_demand[k]));
      }
    }
    __syncthreads();
    // B_k[g] = max over options with at most g GPUs: prefix maximum.
    // budget 0 holds no option (costs are at least 1): T[0] keeps its
    // initial value and the scan runs over budgets 1..G (one pass when G
    // is 64)
    int carry = T[0];
    for (int base = 1; base <= G; base += kWave) {
      const int g = base + lane;
      int v = (g <= G) ? T[g] : INT_MIN;
      v = max(wave_scan_max(v, lane), carry);
      if (g <= G) T[g] = v;
      carry = __shfl(v, kWave - 1, kWave);
    }
    __syncthreads();
    if (k == 0) {
      int *tmp = D; D = T; T = tmp;
    } else if (k + 1 < K) {
      // both tables are nondecreasing in the budget (prefix maxima, and
      // (max,min) convolutions of such), so every target is a crossing search
      // budget 0 is min(D[0], T[0]) (a = 0 only); the others by the search
      if (lane == 0) Dn[0] = min(D[0], T[0]);
      for (int g = 1 + lane; g <= G; g += kWave) Dn[g] = conv_mono(D, T, g, top);
      __syncthreads();
      int *tmp = D; D = Dn; Dn = tmp;
    } else {
      tau = conv_mono(D, T, G, top);
    }
    __syncthreads();
  }
  if (K == 1) tau = D[G];

  if (alloc) {
    float gp = 0.0f;
    for (int k = 0; k < K; ++k) {
      const bool restricted = P.has_floor && floors_met && (P.floor_rps[k] > 0.0f);
      int ti_sel = -1, r_sel = 0;
      if (restricted || tau > 0) {
        // fewest GPUs reaching tau, then the smallest TP index
        int key = INT_MAX;
        for (int ti = 0; ti < P.NT; ++ti) {
          const int t = P.tp[ti];
          for (int r = 1 + lane; t * r <= G; r += kWave) {
            const int b = bmap[k * (G + 1) + r];
            if (b < 0) continue;
            const int cell = cell_of(P, k, ti, b);
            const float c = R.c(cell), l = R.l(cell);
            if (restricted && !floor_ok(c, l, r, P.slo[k], P.demand[k], P.floor_rps[k])) continue;
            if (ratio_bits(c, l, r, P.slo[k], P.rcp_demand[k]) < tau) continue;
            key = min(key, (t * r) * 16 + ti);
          }
        }
        key = wave_min(key);
        if (key != INT_MAX) {
          ti_sel = key & 15;
          r_sel = (key >> 4) / P.tp[ti_sel];
        }
      }
      if (lane == 0) {
        alloc->tp_index[k] = ti_sel;
        alloc->replicas[k] = r_sel;
        if (r_sel > 0) {
          const int cell = cell_of(P, k, ti_sel, bmap[k * (G + 1) + r_sel]);
          gp += served_rps(R.c(cell), r_sel, P.demand[k]);
        }
      }
    }
    if (lane == 0) *goodput = gp;
    __syncthreads();
  }
  return tau;
}

__device__ __forceinline__ void write_alloc(const AllocOut &out, int64_t j, int K, int tau,
                                            int floors_met, float goodput, const WaveAlloc &wa) {
  const int lane = threadIdx.x & (kWave - 1);
  if (lane == 0) {
    if (out.objective) out.objective[j] = __int_as_float(tau);
    if (out.floors_met) out.floors_met[j] = (uint8_t)floors_met;
    if (out.goodput) out.goodput[j] = goodput;
  }
  for (int k = lane; k < K; k += kWave) {
    if (out.tp_index) out.tp_index[j * K + k] = wa.tp_index[k] < 0 ? 0xFF : (uint8_t)wa.tp_index[k];
    if (out.replicas) out.replicas[j * K + k] = (uint16_t)wa.replicas[k];
  }
}

// ---------------------------------------------------------------------------
// LDS staging of a wave solve's inputs.  The solver looks up the bucket map
// and the realisation's cells inside its loops; from global memory every
// lookup is a dependent round trip.  When they fit, the kernels copy the
// bucket map (K (G + 1) bytes) and the realisation's cells (2 N floats)
// into LDS once, with the whole wavefront, and the solver reads them there.
// ---------------------------------------------------------------------------
constexpr size_t kStageLimit = 48 * 1024;  // LDS a staged solve block may use

__device__ __host__ inline size_t stage_bytes(const DevProblem &P) {  // 16: aligning the start
  return 16 + (((size_t)P.K * (P.G + 1) + 3) & ~(size_t)3) + 2 * sizeof(float) * (size_t)P.N;
}

// Whether a solve block stages its inputs: its LDS with the staging area
// stays within kStageLimit.
inline bool stage_fits(size_t lds) { return lds <= kStageLimit; }

struct StageArea {
  int8_t *bmap;
  float *cap, *tail;
};

// p rounded up to a 16-byte boundary.  The pointer stays derived from p (an
// offset added, not an integer turned back into a pointer), so the compiler
// still sees LDS and emits LDS instructions rather than flat ones.
__device__ __forceinline__ char *align16(void *p) {
  char *c = reinterpret_cast<char *>(p);
  return static_cast<char *>(__builtin_assume_aligned(c + ((16 - ((uintptr_t)c & 15)) & 15), 16));
}

__device__ __forceinline__ StageArea stage_area(const DevProblem &P, void *start) {
  StageArea A;
  A.bmap = reinterpret_cast<int8_t *>(align16(start));
  A.cap = reinterpret_cast<float *>(A.bmap + (((size_t)P.K * (P.G + 1) + 3) & ~(size_t)3));
  A.tail = A.cap + P.N;
  return A;
}

__device__ __forceinline__ void stage_copy_bmap(const DevProblem &P, const int8_t *__restrict__ g, int8_t *d) {
  const int n = P.K * (P.G + 1);
  for (int x = threadIdx.x; x < n; x += blockDim.x) d[x] = g[x];
}

__device__ __forceinline__ void stage_copy_cells(const DevProblem &P, const float *__restrict__ gc,
                                                 const float *__restrict__ gt, float *dc, float *dt) {
  for (int x = threadIdx.x; x < P.N; x += blockDim.x) {
    dc[x] = gc[x];
    dt[x] = gt[x];
  }
}

// ---------------------------------------------------------------------------
// Dense batch solve: one wavefront per scenario.
// ---------------------------------------------------------------------------
// STAGE: inputs staged in LDS (1) or read from global memory (0), fixed at
// compile time so that every access compiles for its own memory.
template <int STAGE>
__global__ __launch_bounds__(64) void k_solve_dense(DevProblem P, const int8_t *__restrict__ bmap,
                                                    const float *__restrict__ cap,
                                                    const float *__restrict__ tail, int64_t n,
                                                    AllocOut out) {
  constexpr int stage = STAGE;
  extern __shared__ int lds[];
  const int64_t j = blockIdx.x;
  if (j >= n) return;
  int *tp_index = lds + 3 * (P.G + 1);
  int *replicas = tp_index + kMaxClasses;
  WaveAlloc wa{tp_index, replicas};
  Realisation R{cap + j * P.N, tail + j * P.N, -1, 0.0f, 0.0f};
  if (stage) {
    const StageArea A = stage_area(P, replicas + kMaxClasses);
    stage_copy_bmap(P, bmap, A.bmap);
    stage_copy_cells(P, R.cap, R.tail, A.cap, A.tail);
    bmap = A.bmap;
    R.cap = A.cap;
    R.tail = A.tail;
    __syncthreads();
  }
  int fm;
  float gp;
  const int tau = wave_solve(P, bmap, R, lds, &fm, &wa, &gp);
  write_alloc(out, j, P.K, tau, fm, gp, wa);
}

// ---------------------------------------------------------------------------
// Base realisations of each order: tau(conservative), tau(optimistic).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_base(DevProblem P, const int8_t *__restrict__ bmap,
                                             const float *__restrict__ cap_lo,
                                             const float *__restrict__ cap_hi,
                                             const float *__restrict__ tail_lo,
                                             const float *__restrict__ tail_hi,
                                             int32_t *__restrict__ base) {
  extern __shared__ int lds[];
  const int R = blockIdx.x, o = blockIdx.y;
  const size_t off = (size_t)o * P.N;
  // Section 4.1: conservative = (low capacity, high tail); optimistic = (high, low).
  Realisation real = R == 0 ? Realisation{cap_lo + off, tail_hi + off, -1, 0.0f, 0.0f}
                            : Realisation{cap_hi + off, tail_lo + off, -1, 0.0f, 0.0f};
  int fm;
  const int tau = wave_solve(P, bmap, real, lds, &fm, nullptr, nullptr);
  if (threadIdx.x == 0) base[o * 2 + R] = tau;
}

// ---------------------------------------------------------------------------
// Scores, wave per scenario: block (chunk, e, o) handles samples
// [64*chunk, 64*chunk + 64) one after another; lane j keeps Gamma of sample j.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_score_wave(DevProblem P, const int8_t *__restrict__ bmap,
                                                   const CandInfo *__restrict__ info,
                                                   const float *__restrict__ cap_lo,
                                                   const float *__restrict__ cap_hi,
                                                   const float *__restrict__ tail_lo,
                                                   const float *__restrict__ tail_hi,
                                                   const uint8_t *__restrict__ measured,
                                                   const float *__restrict__ cap_s,
                                                   const float *__restrict__ tail_s, int32_t E,
                                                   int32_t S, const int32_t *__restrict__ base,
                                                   double *__restrict__ partial, int64_t n_partial,
                                                   float *__restrict__ tau_dump) {
  extern __shared__ int lds[];
  const int chunk = blockIdx.x, e = blockIdx.y, o = blockIdx.z;
  const int lane = threadIdx.x;
  const CandInfo ci = info[e];
  const size_t tile = (size_t)o * E + e;
  const size_t off = (size_t)o * P.N;
  if (ci.cls < 0) return;
  if (measured[off + ci.cell]) {
    // nothing to learn from a revealed cell: not solved, score 0
    const int s = chunk * kWave + lane;
    if (tau_dump && s < S) {
      tau_dump[(tile * S + s) * 2 + 0] = __int_as_float(base[o * 2 + 0]);
      tau_dump[(tile * S + s) * 2 + 1] = __int_as_float(base[o * 2 + 1]);
    }
    return;
  }
  double mine = 0.0;
  const int s0 = chunk * kWave;
  const int ns = min(kWave, S - s0);
  for (int j = 0; j < ns; ++j) {
    const float cs = cap_s[tile * S + s0 + j];
    const float ts = tail_s[tile * S + s0 + j];
    int fm;
    Realisation rm{cap_lo + off, tail_hi + off, ci.cell, cs, ts};
    const int tm = wave_solve(P, bmap, rm, lds, &fm, nullptr, nullptr);
    Realisation rp{cap_hi + off, tail_lo + off, ci.cell, cs, ts};
    const int tp = wave_solve(P, bmap, rp, lds, &fm, nullptr, nullptr);
    if (lane == j) mine = (double)__int_as_float(tp) - (double)__int_as_float(tm);
    if (tau_dump && lane == 0) {
      tau_dump[(tile * S + s0 + j) * 2 + 0] = __int_as_float(tm);
      tau_dump[(tile * S + s0 + j) * 2 + 1] = __int_as_float(tp);
    }
  }
  const double sum = wave_pairwise_sum(mine);
  if (lane == 0) partial[tile * n_partial + chunk] = sum;
}

// ---------------------------------------------------------------------------
// Scores, lane per scenario.  Option p of class k enumerates (TP index ti,
// replicas r) as p = off(ti) + r - 1 with off = 0, G, G + G/2, G + G/2 + G/4.
// ---------------------------------------------------------------------------
template <int G>
struct LaneShape {
  static constexpr int PP = G + G / 2 + G / 4 + G / 8;
  static constexpr int off(int ti) {
    return ti == 0 ? 0 : ti == 1 ? G : ti == 2 ? G + G / 2 : G + G / 2 + G / 4;
  }
};

// Per order and realisation, the (cap, tail) every option reads: a gather of
// the order's cells through the load-level map.  Missing options read a zero
// capacity, whose ratio is 0.
template <int G>
__global__ void k_gather_options(DevProblem P, const int8_t *__restrict__ bmap,
                                 const float *__restrict__ cap_lo, const float *__restrict__ cap_hi,
                                 const float *__restrict__ tail_lo,
                                 const float *__restrict__ tail_hi, float *__restrict__ opts) {
  constexpr int PP = LaneShape<G>::PP;
  const int p = threadIdx.x;
  const int k = blockIdx.x, R = blockIdx.y, o = blockIdx.z;
  if (p >= PP) return;
  int ti = 0;
  while (ti < 3 && p >= LaneShape<G>::off(ti + 1)) ++ti;
  const int r = p - LaneShape<G>::off(ti) + 1;
  const int b = bmap[k * (G + 1) + r];
  float c = 0.0f, l = 0.0f;
  if (b >= 0) {
    const size_t cell = (size_t)o * P.N + cell_of(P, k, ti, b);
    c = R == 0 ? cap_lo[cell] : cap_hi[cell];
    l = R == 0 ? tail_hi[cell] : tail_lo[cell];
  }
  const size_t dst = ((((size_t)o * 2 + R) * P.K + k) * PP + p);
  opts[dst * 2 + 0] = c;
  opts[dst * 2 + 1] = l;
}

// B[g-1] = best ratio with at most g GPUs, before the prefix maximum: every
// option max-merged into the slot of its exact GPU count.
template <int G, bool kCandClass>
__device__ __forceinline__ void lane_table(int (&T)[G], const float *__restrict__ opt, float slo,
                                           double rcp, int te, int rlo, int rhi, float cs, float ls) {
#pragma unroll
  for (int g = 0; g < G; ++g) T[g] = 0;
#pragma unroll
  for (int ti = 0; ti < 4; ++ti) {
#pragma unroll
    for (int r = 1; r <= (G >> ti); ++r) {
      const int p = LaneShape<G>::off(ti) + r - 1;
      float c = opt[2 * p], l = opt[2 * p + 1];
      if (kCandClass) {
        const bool sampled = (ti == te) & (r >= rlo) & (r <= rhi);
        c = sampled ? cs : c;
        l = sampled ? ls : l;
      }
      const int f = ratio_bits(c, l, r, slo, rcp);
      T[(r << ti) - 1] = max(T[(r << ti) - 1], f);
    }
  }
#pragma unroll
  for (int g = 1; g < G; ++g) T[g] = max(T[g], T[g - 1]);
}

// D <- D (max,min) T in place.  Entries are budgets 1..G; budget 0 is 0 in
// both, so the a = 0 and a = g terms are 0 and every other term is >= 0.
// Targets run downwards so D[g - a] (a >= 1) is still the old value.
template <int G>
__device__ __forceinline__ void lane_conv(int (&D)[G], const int (&T)[G]) {
#pragma unroll
  for (int g = G; g >= 2; --g) {
    int acc = min(D[g - 2], T[0]);
#pragma unroll
    for (int a = 2; a <= g - 1; ++a) acc = max(acc, min(D[g - a - 1], T[a - 1]));
    D[g - 1] = acc;
  }
  D[0] = 0;
}

template <int G>
__device__ __forceinline__ int lane_final(const int (&D)[G], const int (&T)[G]) {
  int acc = min(D[G - 2], T[0]);
#pragma unroll
  for (int a = 2; a <= G - 1; ++a) acc = max(acc, min(D[G - a - 1], T[a - 1]));
  return acc;
}

template <int G>
__global__ __launch_bounds__(256) void k_score_lane(DevProblem P, const CandInfo *__restrict__ info,
                                                    const uint8_t *__restrict__ measured,
                                                    const float *__restrict__ opts,
                                                    const float *__restrict__ cap_s,
                                                    const float *__restrict__ tail_s, int32_t E,
                                                    int32_t S, const int32_t *__restrict__ base,
                                                    double *__restrict__ partial,
                                                    int64_t n_partial,
                                                    float *__restrict__ tau_dump) {
  constexpr int PP = LaneShape<G>::PP;
  __shared__ double wsum[4];
  const int chunk = blockIdx.x, e = blockIdx.y, o = blockIdx.z;
  const int s = chunk * 256 + threadIdx.x;
  const CandInfo ci = info[e];
  const size_t tile = (size_t)o * E + e;
  if (ci.cls < 0) return;
  if (measured[(size_t)o * P.N + ci.cell]) {
    if (tau_dump && s < S) {
      tau_dump[(tile * S + s) * 2 + 0] = __int_as_float(base[o * 2 + 0]);
      tau_dump[(tile * S + s) * 2 + 1] = __int_as_float(base[o * 2 + 1]);
    }
    return;
  }
  const bool live = s < S;
  float cs = 0.0f, ls = 0.0f;
  if (live) {
    cs = cap_s[tile * S + s];
    ls = tail_s[tile * S + s];
  }
  const int K = P.K;
  int tau_m = 0, tau_p = 0;
#pragma unroll 1
  for (int R = 0; R < 2; ++R) {
    const float *opt = opts + (((size_t)o * 2 + R) * K) * PP * 2;
    int D[G], T[G];
    int tau = 0;
#pragma unroll 1
    for (int k = 0; k < K; ++k) {
      const float *ok = opt + (size_t)k * PP * 2;
      if (k == ci.cls)
        lane_table<G, true>(T, ok, P.slo[k], P.rcp_demand[k], ci.ti, ci.rlo, ci.rhi, cs, ls);
      else
        lane_table<G, false>(T, ok, P.slo[k], P.rcp_demand[k], 0, 1, 0, 0.0f, 0.0f);
      if (k == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) D[g] = T[g];
      } else if (k + 1 < K) {
        lane_conv<G>(D, T);
      } else {
        tau = lane_final<G>(D, T);
      }
    }
    if (K == 1) tau = D[G - 1];
    if (R == 0) tau_m = tau;
    else tau_p = tau;
  }
  double gam = 0.0;
  if (live) {
    gam = (double)__int_as_float(tau_p) - (double)__int_as_float(tau_m);
    if (tau_dump) {
      tau_dump[(tile * S + s) * 2 + 0] = __int_as_float(tau_m);
      tau_dump[(tile * S + s) * 2 + 1] = __int_as_float(tau_p);
    }
  }
  gam = wave_pairwise_sum(gam);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) wsum[w] = gam;
  __syncthreads();
  if (threadIdx.x == 0) {
    // 256 samples per block = four 64-sample blocks of the pairwise tree
    partial[tile * n_partial + chunk] = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
  }
}


// ---------------------------------------------------------------------------
// Exclusion scorer.  The (max,min) convolution is associative and
// commutative, so tau* = (B'_i (.) H_i)[G] where B'_i is the table of the
// candidate's class i and H_i the convolution of every other class.  A
// scenario changes only the candidate's cell, i.e. the options (t, r) with
// r in [rlo, rhi].  With Bx the class-i table without those options and
// f_r the sampled ratio of r replicas, distributivity of min over max gives
//   tau = max( max_g min(Bx[g], H_i[G-g]),  max_r min(f_r, H_i[G - t*r]) )
// (H_i is nondecreasing, so the best budget left for a sampled option of
// cost t*r is all of G - t*r).  The first term, U, and every H_i[G - t*r]
// are per (order, candidate); a scenario costs one ratio and two (max,min)
// steps per replica count in [rlo, rhi].  The result is the same maximum
// over the same binary32 values, so it is bit-identical to the full solve.
// ---------------------------------------------------------------------------

struct Pick {
  double score;
  int tp, cell, e;  // e < 0: nothing
};

__device__ __forceinline__ bool better(const Pick &a, const Pick &b) {
  if (a.e < 0) return false;
  if (b.e < 0) return true;
  if (a.score != b.score) return a.score > b.score;
  if (a.tp != b.tp) return a.tp < b.tp;
  if (a.cell != b.cell) return a.cell < b.cell;
  return a.e < b.e;
}

template <int kCtrl>
__device__ __forceinline__ Pick dpp_pick(const Pick &p) {
  Pick q;
  q.score = dpp_f64<kCtrl>(p.score);
  q.tp = __builtin_amdgcn_mov_dpp(p.tp, kCtrl, 0xF, 0xF, true);
  q.cell = __builtin_amdgcn_mov_dpp(p.cell, kCtrl, 0xF, 0xF, true);
  q.e = __builtin_amdgcn_mov_dpp(p.e, kCtrl, 0xF, 0xF, true);
  return q;
}

__device__ __forceinline__ Pick readlane_pick(const Pick &p, int l) {
  Pick q;
  q.score = readlane_f64(p.score, l);
  q.tp = __builtin_amdgcn_readlane(p.tp, l);
  q.cell = __builtin_amdgcn_readlane(p.cell, l);
  q.e = __builtin_amdgcn_readlane(p.e, l);
  return q;
}

// Best pick of the wavefront (`better` is a strict total order on picks with
// e >= 0, so the combination order does not matter): DPP steps within rows
// of 16 lanes, then the four row winners.  The result is the same in every
// lane.
__device__ __forceinline__ Pick wave_best(Pick p) {
  Pick q = dpp_pick<0xB1>(p);  // quad_perm [1, 0, 3, 2]
  if (better(q, p)) p = q;
  q = dpp_pick<0x4E>(p);  // quad_perm [2, 3, 0, 1]
  if (better(q, p)) p = q;
  q = dpp_pick<0x141>(p);  // row_half_mirror
  if (better(q, p)) p = q;
  q = dpp_pick<0x140>(p);  // row_mirror
  if (better(q, p)) p = q;
  Pick best = readlane_pick(p, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) {
    q = readlane_pick(p, 16 * r);
    if (better(q, best)) best = q;
  }
  return best;
}

// Z[g] = max_{a <= g} min(X[g - a], Y[a]) for one target g.
__device__ __forceinline__ int conv_at(const int *X, const int *Y, int g) {
  int best = INT_MIN;
  for (int a = 0; a <= g; ++a) best = max(best, min(X[g - a], Y[a]));
  return best;
}

// The same target split over 4 consecutive lanes (lane j of the group takes
// a = j, j + 4, ...); every lane of the group returns the full maximum.
// All 64 lanes of the wavefront must call it.
__device__ __forceinline__ int conv_at4(const int *X, const int *Y, int g, bool active) {
  const int j = threadIdx.x & 3;
  int best = INT_MIN;
  if (active) {
#pragma unroll 4
    for (int a = j; a <= g; a += 4) best = max(best, min(X[g - a], Y[a]));
  }
  best = max(best, __shfl_xor(best, 1, kWave));
  best = max(best, __shfl_xor(best, 2, kWave));
  return best;
}

__device__ __forceinline__ double load_acquire(const double *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Pairwise tree over x[0..n), zero-padded to a power of two P2 <= 4096, by
// one full wavefront: lane l first sums its aligned block of P2/64 values
// (a balanced tree in registers), then the lanes combine by butterfly.
__device__ double wave_tree_sum(const double *x, int64_t n) {
  constexpr int kMaxL = 64;
  const int lane = threadIdx.x & (kWave - 1);
  int64_t p2 = 1;
  while (p2 < n) p2 <<= 1;
  const int L = p2 >= kWave ? (int)(p2 / kWave) : 1;
  double v[kMaxL];
#pragma unroll
  for (int j = 0; j < kMaxL; ++j) {
    const int64_t i = (int64_t)lane * L + j;
    v[j] = (j < L && i < n) ? load_acquire(x + i) : 0.0;
  }
#pragma unroll
  for (int w = 1; w < kMaxL; w <<= 1) {
    if (w < L) {
#pragma unroll
      for (int j = 0; j + w < kMaxL; j += 2 * w) v[j] = v[j] + v[j + w];
    }
  }
  return wave_pairwise_sum(v[0]);
}

// Decodes a flattened option index p (0 <= p < P = sum_t floor(G / t)) of
// one class into (TP index, replicas); options are ordered by TP, then r.
__device__ __forceinline__ void option_of(const DevProblem &P, int p, int *ti, int *r) {
  int t = 0;
  for (; t < P.NT - 1; ++t) {
    const int n = P.G / P.tp[t];
    if (p < n) break;
    p -= n;
  }
  *ti = t;
  *r = p + 1;
}

// Smallest binary32 capacity x >= 0 at which r replicas reach ratio bits M,
// i.e. min(1, fl32(fl32(r * x) / demand)) >= M.  The ratio is nondecreasing
// in x and nonnegative binary32 values order like their bit patterns.  The
// quotient M * demand / r lands within a few units in the last place, so the
// eight bit patterns from 3 below it are tested at once (independent
// evaluations, whose latencies overlap): when the first does not reach M
// (or is 0) and the last does, the answer is the first that does.  Otherwise
// the answer is pinned by stepping from the estimate, then by a bisection
// over all bit patterns.  `mode` selects where the search starts: 0 the
// window, 1 the stepping, 2 the bisection (every mode returns the same
// value; 1 and 2 exist so that the later stages can be tested).  0 when
// M <= 0 (always reached); NaN when M exceeds 1 (never reached).
__device__ __forceinline__ float capacity_threshold(int r, int M, float demand, double rcp, int mode) {
  if (M <= 0) return 0.0f;
  if (M > __float_as_int(1.0f)) return __builtin_nanf("");
  const float rf = (float)r;
  auto reach = [&](unsigned xb) {
    const float capacity = rf * __uint_as_float(xb);
    return __float_as_int(fminf((float)((double)capacity * rcp), 1.0f)) >= M;
  };
  unsigned x = __float_as_uint(__int_as_float(M) * demand * __builtin_amdgcn_rcpf(rf));
  if (mode == 0) {
    const unsigned x0 = x > 3u ? x - 3u : 0u;
    int below = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) below += reach(x0 + (unsigned)k) ? 0 : 1;
    if (below < 8 && (below > 0 || x0 == 0u)) return __uint_as_float(x0 + (unsigned)below);
  }
  if (mode <= 1) {
    int n = 0;
    while (!reach(x) && n < 8) { ++x; ++n; }
    while (x > 0 && reach(x - 1) && n < 16) { --x; ++n; }
    if (reach(x) && (x == 0 || !reach(x - 1))) return __uint_as_float(x);
  }
  unsigned blo = 0, bhi = 0x7F800000u;  // +inf reaches ratio 1 >= M
  while (blo < bhi) {
    const unsigned mid = blo + ((bhi - blo) >> 1);
    if (reach(mid)) bhi = mid;
    else blo = mid + 1;
  }
  return __uint_as_float(blo);
}

// Bucket of a replica-range length for the heavy-first work order: longer
// ranges (more work per scenario) get smaller bucket numbers.
__device__ __forceinline__ int range_bucket(int len) { return 31 - min(31, 32 - __clz(len)); }

// Tables of the general set-up's convolution tree: B (K), the first level
// (at least one table: the empty convolution of a single class) and the
// second (the later levels reuse them).
__device__ __host__ inline int prep_tree_a(int K) { return K - 1 > 2 ? (K - 1 + 1) / 2 : 1; }
__device__ __host__ inline int prep_tree_b(int K) { return prep_tree_a(K) > 1 ? (prep_tree_a(K) + 1) / 2 : 1; }

// Problem constants the set-up indexes per lane, staged in LDS (kernel
// arguments are reached through memory loads).
struct PrepConsts {
  float levels[kMaxLevels];
  float demand[kMaxClasses];
  int tp[kMaxTp];
  int optoff[kMaxTp + 1];  // first option of each TP among a class's options
};

// Replica range of a cell: the r in [1, G / t] at the cell's level.  The
// level is nonincreasing in r ("none" sits above every level), so the range
// is [first r at level <= b, first r at level <= b - 1), both by bisection on
// demand / r <= levels[j] (the four argument values are read once).
__device__ __forceinline__ int first_r_at_most(float demand, float level, int rmax) {
  int lo = 1, hi = rmax + 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (demand / (float)mid <= level) hi = mid;
    else lo = mid + 1;
  }
  return lo;
}

__device__ __forceinline__ void cell_range(const DevProblem &P, int cell, int *rlo, int *rhi) {
  const int k = cell / (P.NT * P.B), ti = (cell / P.B) % P.NT, b = cell % P.B;
  const int rmax = P.G / P.tp[ti];
  const float demand = P.demand[k], lb = P.levels[b], lb1 = P.levels[b > 0 ? b - 1 : 0];
  *rlo = first_r_at_most(demand, lb, rmax);
  *rhi = b == 0 ? rmax : first_r_at_most(demand, lb1, rmax) - 1;
}

// Candidate record e: class, TP index and degree, and the replica range
// whose load level is the cell's (1, 0 when none; by bisection, from the
// problem alone, so that it does not wait for the bucket map).
__device__ __forceinline__ void setup_cand_at(const DevProblem &P, const int32_t *__restrict__ cand, int32_t E,
                                              CandInfo *__restrict__ info, int e) {
  if (e >= E) return;
  const int cell = cand[e];
  CandInfo ci;
  ci.cell = cell;
  ci.pad0 = ci.pad1 = 0;
  if (cell < 0 || cell >= P.N) {
    ci.cls = -1; ci.ti = 0; ci.rlo = 1; ci.rhi = 0; ci.tp = 0;
    info[e] = ci;
    return;
  }
  const int ti = (cell / P.B) % P.NT;
  int rlo, rhi;
  cell_range(P, cell, &rlo, &rhi);
  if (rlo > rhi) {
    rlo = 1;
    rhi = 0;
  }
  ci.cls = cell / (P.B * P.NT); ci.ti = ti; ci.rlo = rlo; ci.rhi = rhi; ci.tp = P.tp[ti];
  info[e] = ci;
}

// The scorer's work list (built by one extra block of the set-up): every
// tile the scorer visits -- unrevealed (order, candidate) pairs with a
// nonempty replica range, or every valid pair when dumping -- over all
// orders, longest range first (bucketed by bit length), then end markers up
// to O x E entries.  An entry is self-contained: (candidate, option offset
// of rlo, rlo | nr << 16, class | state << 6 | order << 8).  Also the tile
// records of invalid candidates.  Depends only on the problem and the
// revealed flags.  The order of entries within a bucket is arbitrary (it
// decides only which wavefront evaluates a tile).
__device__ void prep_list(const DevProblem &P, int O, const uint8_t *__restrict__ measured,
                          const int32_t *__restrict__ cand, int E, int dump, int PPc, const PrepConsts &C,
                          TileInfo *__restrict__ tiles, int4 *__restrict__ list, int32_t *__restrict__ n_listed,
                          int *bucket_count, int *bucket_start, int *n_live) {
  const int tid = threadIdx.x, nth = blockDim.x, lane = tid & (kWave - 1);
  const int N = P.N, per_class = P.NT * P.B;
  // Threads work candidate by candidate (the replica range is computed once
  // per candidate); when there are fewer candidates than threads, g threads
  // share a candidate and take every g-th order.  The revealed flags of a
  // candidate's orders are independent loads.
  const int g = E < nth ? nth / E : 1;
  const int sub = E < nth ? tid / E : 0;
  const int e_first = E < nth ? tid - sub * E : tid, e_step = E < nth ? E : nth;
  const bool active = sub < g;
  for (int pass = 0; pass < 2; ++pass) {
    for (int e = e_first; active && e < E; e += e_step) {
      const int cell = cand[e];
      if (cell < 0 || cell >= N) {
        if (pass == 0) {
          for (int o = sub; o < O; o += g) {
            TileInfo *tl = tiles + (size_t)o * E + e;
            tl->state = -1; tl->cell = cell; tl->cls = 0; tl->t = 0; tl->rlo = 1; tl->rhi = 0;
            tl->toff = 0; tl->u_m = 0; tl->u_p = 0; tl->m_m = 0; tl->m_p = 0;
          }
        }
        continue;
      }
      int rlo, rhi;
      cell_range(P, cell, &rlo, &rhi);
      const int nr = rhi >= rlo ? rhi - rlo + 1 : 0;
      if (!dump && nr == 0) continue;  // never visited
      const int b = range_bucket(nr);
      // this thread's listed tiles of candidate e
      int n = 0;
#pragma unroll 8
      for (int o = sub; o < O; o += g) n += (dump || !measured[(size_t)o * N + cell]) ? 1 : 0;
      if (n == 0) continue;
      if (pass == 0) {
        atomicAdd(&bucket_count[b], n);
      } else {
        int at = atomicAdd(&bucket_start[b], n);
        const int k = cell / per_class, ti = (cell / P.B) % P.NT, r0 = nr > 0 ? rlo : 1;
        const int toff = k * PPc + C.optoff[ti] + r0 - 1;
        for (int o = sub; o < O; o += g) {
          const bool meas = measured[(size_t)o * N + cell] != 0;
          if (dump || !meas) list[at++] = make_int4(e, toff, r0 | (nr << 16), k | ((meas ? 1 : 0) << 6) | (o << 8));
        }
      }
    }
    __syncthreads();
    if (pass == 0) {
      if (tid < kWave) {
        const int cnt = lane < 32 ? bucket_count[lane] : 0;
        int incl = cnt;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
          const int u = __shfl_up(incl, d, kWave);
          if (lane >= d) incl += u;
        }
        if (lane < 32) bucket_start[lane] = incl - cnt;
        if (lane == 31) {
          *n_listed = incl;
          *n_live = incl;
        }
      }
      __syncthreads();
    }
  }
  for (int z = *n_live + tid; z < O * E; z += nth) list[z] = make_int4(-1, 0, 0, 0);
}

// B_k of the general set-up, once per (realisation R, order o, class k):
// every option (t, r) with t r < G max-merged into its exact GPU count, then
// the prefix maximum (best ratio with at most g GPUs, g in [0, G)).  Every
// class block of k_prep reads the tables of the other classes from here
// instead of building them itself.
// Threads per B-table block: 256, or 1024 for budgets of 512 and more
// (about 2,000 options per class at G = 1024: 16 classes over 4 orders,
// step 40.6 -> 37.2 us; at G = 256, 1024 threads cost 4 us).
constexpr int kBtabThreadsSmall = 256, kBtabThreadsLarge = 1024;

template <int kBtabThreads>
__global__ __launch_bounds__(kBtabThreads) void k_prep_btab(DevProblem P, const float *__restrict__ cap_lo,
                                                           const float *__restrict__ cap_hi,
                                                           const float *__restrict__ tail_lo,
                                                           const float *__restrict__ tail_hi,
                                                           int32_t *__restrict__ btab) {
  extern __shared__ int bt_lds[];
  const int R = blockIdx.x, o = blockIdx.y, k = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int G = P.G, B = P.B, NT = P.NT, per_class = NT * B, PP = P.optoff[NT];
  int *T = bt_lds;                                         // [G]
  float *cc = reinterpret_cast<float *>(T + G), *ct = cc + per_class;  // class k's cells
  __shared__ float lv[kMaxLevels];
  __shared__ int s_tp[kMaxTp], s_off[kMaxTp + 1];  // indexed per lane below: staged, not kernel arguments
  const size_t off = (size_t)o * P.N + (size_t)k * per_class;
  const float *gcap = (R == 0 ? cap_lo : cap_hi) + off;
  const float *gtail = (R == 0 ? tail_hi : tail_lo) + off;
  for (int g = tid; g < G; g += kBtabThreads) T[g] = 0;  // no option: ratio 0
  for (int c = tid; c < per_class; c += kBtabThreads) {
    cc[c] = gcap[c];
    ct[c] = gtail[c];
  }
  if (tid < B) lv[tid] = P.levels[tid];
  if (tid < NT) s_tp[tid] = P.tp[tid];
  if (tid <= NT) s_off[tid] = P.optoff[tid];
  __syncthreads();
  const float dm = P.demand[k], slo = P.slo[k];
  const double rcp = P.rcp_demand[k];
  for (int q = tid; q < PP; q += kBtabThreads) {
    int ti = 0;
    while (ti + 1 < NT && q >= s_off[ti + 1]) ++ti;
    const int r = q - s_off[ti] + 1, t = s_tp[ti];
    if (t * r >= G) continue;
    const float u = dm / (float)r;
    int lo = 0, hi = B;  // first level >= u; B = none
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (u <= lv[mid]) hi = mid;
      else lo = mid + 1;
    }
    if (lo >= B) continue;
    const int c = ti * B + lo;
    atomicMax(&T[t * r], ratio_bits(cc[c], ct[c], r, slo, rcp));
  }
  __syncthreads();
  // prefix maximum over the block: thread j owns [j L, j L + L); its running
  // maximum, then the maximum of the threads before it (wave scans, then the
  // wavefronts' totals)
  {
    __shared__ int wtot[kBtabThreads / kWave];
    const int L = (G + kBtabThreads - 1) / kBtabThreads;
    int run = 0;
    for (int j = 0; j < L; ++j) {
      const int g = tid * L + j;
      if (g < G) {
        run = max(run, T[g]);
        T[g] = run;
      }
    }
    const int incl = wave_scan_max(run, lane);
    if (lane == kWave - 1) wtot[tid >> 6] = incl;
    __syncthreads();
    int carry = __shfl_up(incl, 1, kWave);
    if (lane == 0) carry = 0;
    for (int w = 0; w < (tid >> 6); ++w) carry = max(carry, wtot[w]);
    for (int j = 0; j < L; ++j) {
      const int g = tid * L + j;
      if (g < G) T[g] = max(T[g], carry);
    }
  }
  __syncthreads();
  int32_t *dst = btab + (((size_t)o * 2 + R) * P.K + k) * G;
  for (int g = tid; g < G; g += kBtabThreads) dst[g] = T[g];
}

// Set-up of the exclusion scorer, one block per (realisation R, order o,
// class i), plus blocks with i = K of which (R = 0, o = 0) builds the work
// list of every order and the others return at once; R = 0 is the
// conservative corner (low capacity, high tail) and R = 1 the optimistic one
// (Section 4.1).  Tables over g in [0, G) (G itself is never read):
//   B_k[g]  best ratio of class k with at most g GPUs (nondecreasing)
//   H_i     the (max,min) convolution of B_k over every k != i, by a tree
// Every (max,min) target of nondecreasing tables is a crossing search.  Then,
// per option o = (TP t, r) of class i on cell c: M_o = H_i[G - t r],
// w_o = min(f_o, M_o), the capacity threshold of M_o, and the cell maximum of
// w_o.  The objective is max(0, max_o w_o) over the options of any one class;
// U(cell) is that maximum over the other cells of the cell's class.  Each
// block writes the tile records of its class's candidates.
//
// Dynamic LDS: all cells (cap, tail) of this realisation; the class's cell
// maxima and replica ranges; the load-level table (K x G int8); and, when
// kLds, the tables (B and two tree buffers, 3 x K x G ints), else in gtab.
__device__ void prep_list_staged(const DevProblem &P, int O, const uint8_t *__restrict__ measured,
                                 const int32_t *__restrict__ cand, int E, int dump, int PPc,
                                 TileInfo *__restrict__ tiles, int4 *__restrict__ list,
                                 int32_t *__restrict__ n_listed, int *lds);

template <bool kLds, int kThreads>
__global__ __launch_bounds__(kThreads) void k_prep(DevProblem P, const float *__restrict__ cap_lo,
                                             const float *__restrict__ cap_hi,
                                             const float *__restrict__ tail_lo,
                                             const float *__restrict__ tail_hi,
                                             const uint8_t *__restrict__ measured,
                                             const int32_t *__restrict__ cand, int32_t E, int32_t dump,
                                             int32_t *__restrict__ gtab, TileInfo *__restrict__ tiles,
                                             int32_t *__restrict__ base, int32_t *__restrict__ mopt,
                                             float *__restrict__ thr, int32_t n_thr,
                                             int4 *__restrict__ list, int32_t *__restrict__ n_listed,
                                             int32_t thr_mode, int32_t staged_list,
                                             const int32_t *__restrict__ btab) {
  extern __shared__ int lds[];
  __shared__ PrepConsts C;
  __shared__ int bucket_count[32], bucket_start[32], n_live;
  const int R = blockIdx.x, o = blockIdx.y, ci = blockIdx.z;
  const int tid = threadIdx.x, nth = blockDim.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & (kWave - 1);
  const int G = P.G, K = P.K, N = P.N, NT = P.NT, B = P.B, KG = K * G;
  const int per_class = NT * B;
  const int PPc = n_thr / K;
  if (tid < NT) C.tp[tid] = P.tp[tid];
  if (tid == 0) {
    int at = 0;
    for (int t = 0; t < NT; ++t) {
      C.optoff[t] = at;
      at += G / P.tp[t];
    }
    C.optoff[NT] = at;
  }
  if (ci == K) {  // one block builds the work list of every order
    if (R != 0 || o != 0) return;
    if (staged_list) {
      prep_list_staged(P, (int)gridDim.y, measured, cand, E, dump, PPc, tiles, list, n_listed, lds);
      return;
    }
    if (tid < 32) bucket_count[tid] = 0;
    __syncthreads();
    prep_list(P, (int)gridDim.y, measured, cand, E, dump, PPc, C, tiles, list, n_listed, bucket_count,
              bucket_start, &n_live);
    return;
  }
  float *ccap = (float *)lds;                // [N]
  float *ctail = ccap + N;                   // [N]
  int *mc = (int *)(ctail + N);              // [per_class] cell maxima of class ci
  int *crlo = mc + per_class;                // [per_class] replica ranges of class ci
  int *crhi = crlo + per_class;              // [per_class]
  int8_t *lvl = (int8_t *)(crhi + per_class);  // [K][G] load level of r = g + 1 replicas
  int *tabs = kLds ? (int *)(lvl + ((KG + 15) & ~15)) : gtab + (((size_t)o * 2 + R) * K + ci) * 3 * KG;
  int *Bt = tabs;                            // [K][G]
  // tree buffers: [ceil((K-1)/2)][G] and [ceil(ceil((K-1)/2)/2)][G] (the
  // levels of the tree alternate between them, each no wider than the last)
  int *Xa = tabs + KG, *Xb = Xa + prep_tree_a(K) * G;
  const size_t off = (size_t)o * N;
  const float *gcap = (R == 0 ? cap_lo : cap_hi) + off;
  const float *gtail = (R == 0 ? tail_hi : tail_lo) + off;
  int top = 1;
  while (2 * top <= G) top <<= 1;  // 2 * top > G >= g + 1

  // --- stage the cells; each thread's first candidate is read now
  for (int c = tid; c < N; c += nth) {
    ccap[c] = gcap[c];
    ctail[c] = gtail[c];
  }
  for (int c = tid; c < per_class; c += nth) {
    mc[c] = INT_MIN;
    crlo[c] = INT_MAX;
    crhi[c] = -1;
  }
  if (tid < B) C.levels[tid] = P.levels[tid];
  if (tid < K) C.demand[tid] = P.demand[tid];
  const int my_cell = tid < E ? cand[tid] : -1;
  __syncthreads();
  const bool my_valid = my_cell >= 0 && my_cell < N;
  const int my_meas = (R == 0 && my_valid && my_cell / per_class == ci) ? measured[off + my_cell] : 0;

  // --- load level of class ci's replica counts: the smallest level holding
  // demand / r (the other classes enter through their B tables only)
  for (int idx = ci * G + tid; idx < (ci + 1) * G; idx += nth) {
    const int k = ci, r = idx - k * G + 1;
    const float per_replica = C.demand[k] / (float)r;
    int lo = 0, hi = B;  // first level >= per_replica; B = none
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (per_replica <= C.levels[mid]) hi = mid;
      else lo = mid + 1;
    }
    lvl[idx] = (int8_t)(lo < B ? lo : -1);
  }
  __syncthreads();

  // --- B tables of the other classes, built once per (realisation, order)
  // by k_prep_btab: copied into LDS (16-byte moves when they align), or read
  // in place when the tables live in global memory
  const int32_t *gB = btab + ((size_t)o * 2 + R) * (size_t)KG;
  const int *Bsrc = gB;
  if (kLds) {
    if ((KG & 3) == 0 && (reinterpret_cast<uintptr_t>(Bt) & 15) == 0) {
      const int4 *src4 = reinterpret_cast<const int4 *>(gB);
      int4 *dst4 = reinterpret_cast<int4 *>(Bt);
      for (int x = tid; x < KG / 4; x += nth) dst4[x] = src4[x];
    } else {
      for (int x = tid; x < KG; x += nth) Bt[x] = gB[x];
    }
    Bsrc = Bt;
    __syncthreads();
  }

  // --- H_ci: tree over the tables k != ci.  Level 0 reads B (logical table
  // j is class j, or j + 1 from ci on); later levels alternate Xa / Xb.  For
  // nondecreasing tables the (max,min) convolution of two is the first G
  // entries of their ascending merge (Z[g] >= v iff at most g entries of
  // the two lie below v), so a pair is merged: each thread takes `cw`
  // consecutive outputs, finds where they start by a bisection over the
  // split and then takes them one merge step at a time (one read per step,
  // where a bisection per output reads 2 log2 G entries).
  const int n0 = K - 1;
  const int *H;
  if (K == 1) {
    for (int g = tid; g < G; g += nth) Xa[g] = INT_MAX;  // the empty convolution
    H = Xa;
    __syncthreads();
  } else if (n0 == 1) {
    H = Bsrc + (ci == 0 ? 1 : 0) * G;
  } else {
    int n = n0;
    int *src = nullptr, *dst = Xa;
    while (n > 1) {
      const int pairs = n >> 1, odd = n & 1;
      // outputs per thread: enough that the pairs fill the block, at least 4
      int cw = (pairs * G + nth - 1) / nth;
      cw = cw < 4 ? 4 : cw;
      const int per = (G + cw - 1) / cw;
      for (int item = tid; item < pairs * per; item += nth) {
        const int p = item / per, c0 = (item - p * per) * cw;
        const int ja = 2 * p, jb = 2 * p + 1;
        const int *X = src ? src + ja * G : Bsrc + (ja < ci ? ja : ja + 1) * G;
        const int *Y = src ? src + jb * G : Bsrc + (jb < ci ? jb : jb + 1) * G;
        int i = merge_split(X, Y, G, c0), j = c0 - i;
        int xv = X[min(i, G - 1)], yv = Y[min(j, G - 1)];
        const int c1 = min(c0 + cw, G);
        for (int g = c0; g < c1; ++g) {
          const bool take_x = i < G && (j >= G || xv <= yv);
          dst[p * G + g] = take_x ? xv : yv;
          if (take_x) {
            ++i;
            xv = X[min(i, G - 1)];
          } else {
            ++j;
            yv = Y[min(j, G - 1)];
          }
        }
      }
      if (odd) {  // the odd table passes through
        const int ja = 2 * pairs;
        const int *X = src ? src + ja * G : Bsrc + (ja < ci ? ja : ja + 1) * G;
        for (int g = tid; g < G; g += nth) dst[pairs * G + g] = X[g];
      }
      __syncthreads();
      n = pairs + odd;
      src = dst;
      dst = dst == Xa ? Xb : Xa;
    }
    H = src;
  }

  // --- options of class ci: M, threshold, and w folded into the cell maximum
  {
    int32_t *Mo = mopt + ((size_t)o * 2 + R) * n_thr + (size_t)ci * PPc;
    float *To = thr + ((size_t)o * 2 + R) * n_thr + (size_t)ci * PPc;
    const float slo = P.slo[ci], demand = P.demand[ci];
    const double rcp = P.rcp_demand[ci];
    // whole wavefronts per pass (the cell folds shuffle across lanes)
    for (int p0 = tid - lane; p0 < PPc; p0 += nth) {
      const int p = p0 + lane;
      int key = -1, w = 0, r = 1;
      if (p < PPc) {
        int ti = 0;
        while (ti + 1 < NT && p >= C.optoff[ti + 1]) ++ti;
        r = p - C.optoff[ti] + 1;
        const int t = C.tp[ti];
        const int b = lvl[ci * G + r - 1];
        if (b < 0) {
          Mo[p] = INT_MIN;
          To[p] = __builtin_nanf("");
        } else {
          const int local = ti * B + b, cell = ci * per_class + local;
          // ratios never exceed 1, so M above 1 acts as 1 (min(f, M) and the
          // crossing are unchanged) and the scorer can skip the clamp of f
          const int M = min(H[G - t * r], __float_as_int(1.0f));
          const int f = ratio_bits(ccap[cell], ctail[cell], r, slo, rcp);
          key = local;
          w = min(f, M);
          Mo[p] = M;
          To[p] = capacity_threshold(r, M, demand, rcp, thr_mode);
        }
      }
      fold_cell_runs(key, w, r, mc, crlo, crhi);
    }
  }
  __syncthreads();

  // --- tile records of class ci's candidates and U; the base objective
  for (int e = tid; e < E; e += nth) {
    const int cell = e == tid ? my_cell : cand[e];
    if (cell < 0 || cell >= N || cell / per_class != ci) continue;
    TileInfo *tl = tiles + (size_t)o * E + e;
    const int local = cell - ci * per_class;
    int u0 = 0, u1 = 0, u2 = 0, u3 = 0;  // the other cells' best, 4 chains
    int c = 0;
    for (; c + 4 <= per_class; c += 4) {
      u0 = max(u0, c + 0 != local ? mc[c + 0] : 0);
      u1 = max(u1, c + 1 != local ? mc[c + 1] : 0);
      u2 = max(u2, c + 2 != local ? mc[c + 2] : 0);
      u3 = max(u3, c + 3 != local ? mc[c + 3] : 0);
    }
    for (; c < per_class; ++c) u0 = max(u0, c != local ? mc[c] : 0);
    const int u = max(max(u0, u1), max(u2, u3));
    const int ti = local / B;
    const int nr = crhi[local] >= crlo[local] ? crhi[local] - crlo[local] + 1 : 0;
    // M at rlo, the same value as the option's
    const int m_lo = nr > 0 ? min(H[G - C.tp[ti] * crlo[local]], __float_as_int(1.0f)) : 0;
    if (R == 0) {
      const int meas = e == tid ? my_meas : measured[off + cell];
      tl->cls = ci; tl->t = C.tp[ti]; tl->cell = cell;
      tl->rlo = nr > 0 ? crlo[local] : 1;
      tl->rhi = nr > 0 ? crhi[local] : 0;
      tl->state = meas ? 1 : 0;
      tl->toff = ci * PPc + C.optoff[ti] + (nr > 0 ? crlo[local] : 1) - 1;
      tl->u_m = u;
      tl->m_m = m_lo;
    } else {
      tl->u_p = u;
      tl->m_p = m_lo;
    }
  }
  if (ci == 0 && wave == 0) {
    int v = 0;  // 0: the empty allocation
    for (int c = lane; c < per_class; c += kWave) v = max(v, mc[c]);
    v = wave_max(v);
    if (lane == 0) base[o * 2 + R] = v;
  }
}

// ---------------------------------------------------------------------------
// Set-up of the exclusion scorer for budgets of at most one wavefront.
// ---------------------------------------------------------------------------
// Largest budget and class count of the one-block-per-order set-up.
constexpr int kPrepOrderMaxG = kWave;
constexpr int kPrepOrderMaxK = 16;

// Load level of every (class k, replica count r) for the set-up with one
// block per order, from the problem statement alone (filled on the host,
// passed by value): lvl[k * kPrepOrderMaxG + r - 1] is the smallest level
// holding lambda_k / r (binary32), -1 when none does.
struct PrepLevels {
  int8_t lvl[kPrepOrderMaxK * kPrepOrderMaxG];
};
// Wavefronts per block of the per-order set-up: one per class, and one per
// 1024 listed tiles (at most 16) so the work-list block has threads enough
// for large lists; a class block's wavefronts beyond K only help stage the
// order (extra wavefronts make its barriers slower, so small lists keep K).
static int prep_order_waves(const DevProblem &P, int64_t O, int64_t E) {
  const int64_t by_list = (O * E + 1023) / 1024;
  const int64_t by_class = 2 * P.K <= 16 ? 2 * P.K : P.K;
  const int64_t w = by_list > by_class ? by_list : by_class;
  return (int)(w < 16 ? w : 16);
}

// The scorer's work list, built by one block from staged inputs: the
// candidates' cells and every order's revealed flags are read into LDS in
// one round trip, during which the block finds, for every (class, level),
// the first and last replica count r in [1, G] whose per-replica load lands
// in that level, by two bisections (the level is nonincreasing in r, so
// these form a range; a cell of TP t keeps the part with t r <= G).  The list holds every tile the
// scorer visits -- an unrevealed (order, candidate) pair whose cell some
// replica count reaches, or every valid pair when dumping -- over all
// orders, longest range first (bucketed by bit length), then end markers up
// to O x E entries.  An entry is self-contained: (candidate, option offset
// of rlo, rlo | nr << 16, class | revealed << 6 | order << 8).  The order of
// entries within a bucket is arbitrary: it decides only which wavefront
// evaluates a tile.  Also writes the tile records of invalid candidates.
//
// LDS: bucket counters and starts (2 x 32 + 4), the level ranges (2 x K x B),
// per candidate its cell and range code (2 x E), the revealed flags (O x N
// bytes).
__device__ void prep_list_staged(const DevProblem &P, int O, const uint8_t *__restrict__ measured,
                                 const int32_t *__restrict__ cand, int E, int dump, int PPc,
                                 TileInfo *__restrict__ tiles, int4 *__restrict__ list,
                                 int32_t *__restrict__ n_listed, int *lds) {
  const int tid = threadIdx.x, nth = blockDim.x, lane = tid & (kWave - 1);
  const int N = P.N, G = P.G, K = P.K, B = P.B, per_class = P.NT * P.B;
  int *bucket_count = lds, *bucket_start = lds + 32, *n_live = lds + 64;
  int *lv_first = lds + 68, *lv_last = lv_first + K * B;
  int *c_cell = lv_last + K * B, *c_code = c_cell + E;
  uint8_t *meas = reinterpret_cast<uint8_t *>(c_code + E);
  __shared__ int c_tp[kMaxTp], c_optoff[kMaxTp + 1];
  if (tid < P.NT) c_tp[tid] = P.tp[tid];
  if (tid <= P.NT) c_optoff[tid] = P.optoff[tid];
  if (tid < 32) bucket_count[tid] = 0;
  stage_u8(meas, measured, O * N, tid, nth);
  for (int e = tid; e < E; e += nth) c_cell[e] = cand[e];
  // every (class, level)'s replica range in [1, G]: the level falls as r
  // grows, so it is [first r at the level or below, first r at the level
  // below) -- two bisections per pair instead of a level per (class, r)
  for (int x = tid; x < K * B; x += nth) {
    const int k = x / B, b = x - k * B;
    const float dm = P.demand[k];
    lv_first[x] = first_r_at_most(dm, P.levels[b], G);
    lv_last[x] = b == 0 ? G : first_r_at_most(dm, P.levels[b - 1], G) - 1;
  }
  __syncthreads();
  // range code of a candidate: -1 invalid cell, -2 never visited (no replica
  // count reaches the cell and nothing is dumped), else r0 | nr << 16
  for (int e = tid; e < E; e += nth) {
    const int cell = c_cell[e];
    int code = -1;
    if (cell >= 0 && cell < N) {
      const int k = cell / per_class, ti = (cell / B) % P.NT, b = cell % B;
      const int rlo = lv_first[k * B + b], rhi = min(lv_last[k * B + b], G / c_tp[ti]);
      const int nr = rhi >= rlo ? rhi - rlo + 1 : 0;
      code = (!dump && nr == 0) ? -2 : ((nr > 0 ? rlo : 1) | (nr << 16));
    }
    c_code[e] = code;
  }
  __syncthreads();
  // Threads work candidate by candidate; when there are fewer candidates
  // than threads, g threads share a candidate and take every g-th order.
  const int g = E < nth ? nth / E : 1;
  const int sub = E < nth ? tid / E : 0;
  const int e_first = E < nth ? tid - sub * E : tid, e_step = E < nth ? E : nth;
  const bool active = sub < g;
  for (int pass = 0; pass < 2; ++pass) {
    for (int e = e_first; active && e < E; e += e_step) {
      const int code = c_code[e], cell = c_cell[e];
      if (code == -1) {
        if (pass == 0) {
          for (int o = sub; o < O; o += g) {
            TileInfo *tl = tiles + (size_t)o * E + e;
            tl->state = -1; tl->cell = cell; tl->cls = 0; tl->t = 0; tl->rlo = 1; tl->rhi = 0;
            tl->toff = 0; tl->u_m = 0; tl->u_p = 0; tl->m_m = 0; tl->m_p = 0;
          }
        }
        continue;
      }
      if (code == -2) continue;
      const int nr = code >> 16, b = range_bucket(nr);
      // the thread's orders o = sub, sub + g, ..., their revealed flags read
      // eight at a time: unconditional reads at clamped orders (an order
      // past O counts as revealed), so the reads of a batch overlap
      auto flags = [&](int o0, uint8_t (&mv)[8]) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int o = o0 + u * g;
          const uint8_t f = meas[min(o, O - 1) * N + cell];
          mv[u] = o < O ? f : 1;
        }
      };
      int n = 0;
      for (int o0 = sub; o0 < O; o0 += 8 * g) {
        uint8_t mv[8];
        flags(o0, mv);
#pragma unroll
        for (int u = 0; u < 8; ++u) n += (o0 + u * g < O && (dump || !mv[u])) ? 1 : 0;
      }
      if (n == 0) continue;
      if (pass == 0) {
        atomicAdd(&bucket_count[b], n);
      } else {
        int at = atomicAdd(&bucket_start[b], n);
        const int k = cell / per_class, ti = (cell / B) % P.NT;
        const int toff = k * PPc + c_optoff[ti] + (code & 0xFFFF) - 1;
        for (int o0 = sub; o0 < O; o0 += 8 * g) {
          uint8_t mv[8];
          flags(o0, mv);
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int o = o0 + u * g;
            const bool rev = mv[u] != 0;
            if (o < O && (dump || !rev)) list[at++] = make_int4(e, toff, code, k | ((rev ? 1 : 0) << 6) | (o << 8));
          }
        }
      }
    }
    // the end markers below need only the count from the first pass: no
    // barrier (and no wait for the list's stores) after the second
    if (pass == 0) {
      __syncthreads();
      if (tid < kWave) {
        const int cnt = lane < 32 ? bucket_count[lane] : 0;
        const int incl = wave_scan_add_rows(cnt, lane);
        if (lane < 32) bucket_start[lane] = incl - cnt;
        if (lane == 31) {
          *n_listed = incl;
          *n_live = incl;
        }
      }
      __syncthreads();
    }
  }
  for (int z = *n_live + tid; z < O * E; z += nth) list[z] = make_int4(-1, 0, 0, 0);
}

// Set-up of the exclusion scorer when the budget fits one wavefront
// (G <= 64) and K <= 16: one block per (order o, realisation R) --
// block 2 o + R -- with one wavefront per class (and idle ones when the
// list is large), and block 2 O builds the work list.  R = 0 is the
// conservative corner (low capacity, high tail), R = 1 the optimistic one
// (Section 4.1).  The same quantities as the
// general set-up, with fewer barriers:
//   1. all threads: the order's cells and candidates into LDS; the load
//      level of every (class, r) (the count of grid levels below
//      lambda / r is the index of the smallest level holding it)
//   2. wavefront k: B_k, the best ratio of class k with at most g GPUs: per
//      budget the options of exactly that cost, then a prefix maximum
//   3. wavefront j: the rank of each value of B_j among the other tables,
//      scattered into every H_i (i != j); H_i, the (max,min) convolution of
//      the tables but B_i, is the prefix maximum of that scatter
//   4. wavefront i, on its own: per option of class i, M = H_i[G - t r]
//      clamped at 1, the capacity threshold of M and w = min(f, M) folded
//      into its cell's maximum; U of each of its candidates from the two
//      largest cell maxima; tile records; the base objective (class 0).
// Tables cover g in [0, G) (option costs t r >= 1 read H at G - t r < G).
//
// LDS of a class block: cells (2N floats), the B tables and the H scatter
// (2 x K x G), the candidates (E), per class wavefront (two per class when
// K <= 8) 3 NT B ints (cell maxima, replica ranges), the order's revealed
// flags (N bytes, padded to 4) and the load levels (K x G bytes).
template <int KP, int NTP>
__global__ __launch_bounds__(1024) void k_prep_order(DevProblem P, const float *__restrict__ cap_lo,
                                                     const float *__restrict__ cap_hi,
                                                     const float *__restrict__ tail_lo,
                                                     const float *__restrict__ tail_hi,
                                                     const uint8_t *__restrict__ measured,
                                                     const int32_t *__restrict__ cand, int32_t E, int32_t O,
                                                     int32_t dump, TileInfo *__restrict__ tiles,
                                                     int32_t *__restrict__ base, int32_t *__restrict__ mopt,
                                                     float *__restrict__ thr, int32_t n_thr,
                                                     int4 *__restrict__ list, int32_t *__restrict__ n_listed,
                                                     int32_t thr_mode, const PrepLevels LV) {
  extern __shared__ int lds[];
  const int tid = threadIdx.x, nth = blockDim.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = P.G, K = P.K, N = P.N, NT = P.NT, B = P.B, per_class = NT * B;
  const int PPc = n_thr / K;
  if ((int)blockIdx.x == 2 * O) {
    prep_list_staged(P, O, measured, cand, E, dump, PPc, tiles, list, n_listed, lds);
    return;
  }
  const int o = blockIdx.x >> 1, R = blockIdx.x & 1;
  float *ccap = reinterpret_cast<float *>(lds);
  float *ctail = ccap + N;
  int *Bt = reinterpret_cast<int *>(ctail + N);  // [K][G] B tables
  int *Hs = Bt + K * G;                          // [K][G] rank scatter of H
  int *ccand = Hs + K * G;                       // [E]
  const int wstride = 3 * per_class;
  // per-wavefront areas: one per class, two when a second wavefront per
  // class computes the thresholds (at most 8 classes)
  const int nwa = (int)(blockDim.x >> 6) >= 2 * K ? 2 * K : K;
  int *wbase = ccand + E;                        // [nwa][wstride]
  uint8_t *mrow = reinterpret_cast<uint8_t *>(wbase + nwa * wstride);  // [N]
  int8_t *lvl = reinterpret_cast<int8_t *>(mrow + ((N + 3) & ~3));   // [K][G]
  int *mc = wbase + wave * wstride, *crlo = mc + per_class, *crhi = crlo + per_class;
  const size_t off = (size_t)o * N;
  const float *gcap = (R == 0 ? cap_lo : cap_hi) + off;
  const float *gtail = (R == 0 ? tail_hi : tail_lo) + off;

  // the TP degrees and option offsets in registers: read unconditionally
  // (a few wide scalar loads), so later loops over TP degrees touch no memory
  int tpr[NTP], ofr[NTP];
  float tpinv[NTP];
#pragma unroll
  for (int j = 0; j < NTP; ++j) {
    tpr[j] = P.tp[j];
    ofr[j] = P.optoff[j];
    tpinv[j] = tpr[j] > 0 ? 1.0f / (float)tpr[j] : 0.0f;
  }

  // --- 1. stage the order; load levels while the loads are in flight
  __shared__ int c_tp[kMaxTp], c_optoff[kMaxTp + 1];
  if (tid < NT) c_tp[tid] = P.tp[tid];
  if (tid <= NT) c_optoff[tid] = P.optoff[tid];
  for (int c = tid; c < N; c += nth) {
    ccap[c] = gcap[c];
    ctail[c] = gtail[c];
    if (R == 0) mrow[c] = measured[off + c];
  }
  for (int e = tid; e < E; e += nth) ccand[e] = cand[e];
  if (wave < K && lane < G) lvl[wave * G + lane] = LV.lvl[wave * kPrepOrderMaxG + lane];  // r = lane + 1
  for (int c = lane; wave < K && c < per_class; c += kWave) {
    mc[c] = INT_MIN;
    crlo[c] = INT_MAX;
    crhi[c] = -1;
  }
  __syncthreads();

  // --- 2. wavefront k: B_k, one lane per budget g < G.  The options of
  // exact cost g are (t, g / t) for the TP degrees t dividing g; each reads
  // its cell from LDS (all reads independent), then a prefix maximum over
  // the lanes.  The table goes to LDS for the other wavefronts and stays in
  // a register; the scatter targets of step 3 are cleared meanwhile.
  int btab = 0;
  if (wave < K) {
    const int k = wave;
    const float slo = P.slo[k];
    const double rcp = P.rcp_demand[k];
    const int g = lane;
    // all reads of a kind issued together: the levels of every (t, g / t),
    // then their cells
    int rr[NTP], bb[NTP];
    bool ok[NTP];
#pragma unroll
    for (int ti = 0; ti < NTP; ++ti) {
      const int t = tpr[ti];
      // g / t, exact whenever t divides g (g < 64, t <= 4096: the float
      // quotient is within 1/2 of it)
      const int r = (int)((float)g * tpinv[ti] + 0.5f);
      ok[ti] = ti < NT && g > 0 && g < G && r >= 1 && r * t == g;
      rr[ti] = ok[ti] ? r : 1;
      bb[ti] = lvl[k * G + rr[ti] - 1];
    }
    __builtin_amdgcn_sched_barrier(0);
    float cc[NTP], ct[NTP];
#pragma unroll
    for (int ti = 0; ti < NTP; ++ti) {
      const int cell = (k * NT + min(ti, NT - 1)) * B + max(bb[ti], 0);
      cc[ti] = ccap[cell];
      ct[ti] = ctail[cell];
    }
    __builtin_amdgcn_sched_barrier(0);
    int best = 0;  // budget 0 and costs no option has: ratio 0
#pragma unroll
    for (int ti = 0; ti < NTP; ++ti) {
      const int f = ratio_bits(cc[ti], ct[ti], rr[ti], slo, rcp);
      best = max(best, ok[ti] && bb[ti] >= 0 ? f : 0);
    }
    btab = wave_scan_max_nonneg(best, lane);
    if (lane < G) {
      Bt[k * G + lane] = btab;
      Hs[k * G + lane] = 0;  // ratio 0: the smallest value a table holds
    }
  }
  __syncthreads();

  // --- 3. H_i, the (max,min) convolution of every table but B_i.  For
  // nondecreasing tables the convolution of two is the first G entries of
  // their sorted merge (H[g] >= v iff the entries below v, counted in both,
  // number at most g), so H_i[g] is the entry of rank g in the union of the
  // other classes' tables: every value v of B_j goes to H_i at index
  // rank_i(v) = (entries below v in every table but B_i), with the largest
  // value per index kept, and a prefix maximum fills the rest.  Wavefront j
  // counts, for each v of its own table (first occurrences only), the
  // entries below v in every table by a bisection over register copies of
  // the tables (cross-lane reads by ds_bpermute, all K searches
  // interleaved), and scatters v into the K - 1 targets.
  if (wave < K && K > 1) {
    const int j = wave;
    // KP >= K tables, those past K empty (INT_MAX: never below v), so that
    // the searches are straight-line code whatever K is
    int tb[KP];
#pragma unroll
    for (int k = 0; k < KP; ++k) {
      const int x = Bt[min(k, K - 1) * G + min(lane, G - 1)];
      tb[k] = k < K && lane < G ? x : INT_MAX;
    }
    const int v = btab;
    const int prev = __builtin_amdgcn_ds_bpermute(4 * (lane > 0 ? lane - 1 : 0), v);
    const bool first = lane < G && (lane == 0 || prev != v);
    int cnt[KP];
#pragma unroll
    for (int k = 0; k < KP; ++k) cnt[k] = 0;
    // cnt counts the entries below v: after the steps 64, 32, ..., 1 it is
    // the first index whose entry is not below v (entries past G are
    // INT_MAX, never below)
#pragma unroll
    for (int step = kWave; step > 0; step >>= 1) {
      int e[KP];
#pragma unroll
      for (int k = 0; k < KP; ++k) e[k] = __builtin_amdgcn_ds_bpermute(4 * min(cnt[k] + step - 1, kWave - 1), tb[k]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int k = 0; k < KP; ++k) cnt[k] += (cnt[k] + step - 1 < kWave && e[k] < v) ? step : 0;
    }
    int tot = 0;
#pragma unroll
    for (int k = 0; k < KP; ++k) tot += cnt[k];
#pragma unroll
    for (int k = 0; k < KP; ++k) {
      const int rank = tot - cnt[k];
      if (k < K && k != j && first && rank < G) atomicMax(&Hs[k * G + rank], v);
    }
  }
  __syncthreads();

  // --- 4. wavefront i on its own from here.  With at most 8 classes a
  // second wavefront per class (K + i) computes the same H_i and only the
  // capacity thresholds, which nothing else in the block needs, so the
  // first one goes on to U and the records without them.
  const bool split = (int)(blockDim.x >> 6) >= 2 * K;
  if (wave >= (split ? 2 * K : K)) return;
  const bool thr_wave = wave >= K;
  const bool do_thr = !split || thr_wave, do_cells = !split || !thr_wave;
  const int i = thr_wave ? wave - K : wave;
  // H_i in a register (lane g: H_i[g]); with one class, the empty
  // convolution (no other class constrains the budget)
  const int hreg = K == 1 ? INT_MAX : wave_scan_max_nonneg(lane < G ? Hs[i * G + lane] : 0, lane);
  {
    int32_t *Mo = mopt + ((size_t)o * 2 + R) * n_thr + (size_t)i * PPc;
    float *To = thr + ((size_t)o * 2 + R) * n_thr + (size_t)i * PPc;
    const float slo = P.slo[i], demand = P.demand[i];
    const double rcp = P.rcp_demand[i];
    // Options two wavefronts' worth at a time: lane l takes options
    // base + l and base + l + 64 together, so their LDS reads and threshold
    // searches overlap (one pass when the class has at most 128 options).
    for (int base = 0; base < PPc; base += 2 * kWave) {
      int rr[2], Mv[2], fv[2], loc[2];
      bool has[2], ok[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int p = base + lane + u * kWave;
        int ti = 0, first = 0, t = tpr[0];
#pragma unroll
        for (int t2 = 1; t2 < NTP; ++t2) {
          const bool in = t2 < NT && p >= ofr[t2];
          ti = in ? t2 : ti;
          first = in ? ofr[t2] : first;
          t = in ? tpr[t2] : t;
        }
        // every read below is at a valid index whether or not the option
        // exists (r = 1 past the last option; level 0 for an option with no
        // level), so the reads are unconditional and overlap
        has[u] = p < PPc;
        const int r = has[u] ? p - first + 1 : 1;
        const int bl = lvl[i * G + r - 1];
        const int b = has[u] ? bl : -1;
        ok[u] = b >= 0;
        const int local = ti * B + (ok[u] ? b : 0), cell = i * per_class + local;
        const int hv = __builtin_amdgcn_ds_bpermute(4 * max(G - t * r, 0), hreg);
        const float cc = ccap[cell], ct = ctail[cell];
        // ratios never exceed 1, so M above 1 acts as 1 (min(f, M) and the
        // crossing are unchanged) and the scorer can skip the clamp of f
        rr[u] = r;
        loc[u] = local;
        Mv[u] = ok[u] ? min(hv, __float_as_int(1.0f)) : INT_MIN;
        fv[u] = ok[u] ? ratio_bits(cc, ct, r, slo, rcp) : 0;
      }
      float Tv[2] = {0.0f, 0.0f};
      if (do_thr) {
#pragma unroll
        for (int u = 0; u < 2; ++u) Tv[u] = ok[u] ? capacity_threshold(rr[u], Mv[u], demand, rcp, thr_mode) : __builtin_nanf("");
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        if (do_cells) fold_cell_runs(ok[u] ? loc[u] : -1, min(fv[u], Mv[u]), rr[u], mc, crlo, crhi);
        const int p = base + lane + u * kWave;
        if (do_thr && has[u]) {
          Mo[p] = Mv[u];
          To[p] = Tv[u];
        }
      }
    }
  }
  if (!do_cells) return;  // the threshold wavefront is done
  wave_lds_fence();
  // U of a cell is the largest maximum among the class's other cells (or 0):
  // the largest maximum m1 at its lowest index c1, and the largest m2 over
  // every other cell, give it for every cell at once
  int m1 = INT_MIN, c1 = INT_MAX;
  for (int c = lane; c < per_class; c += kWave) {
    const int v = mc[c];
    if (v > m1) {
      m1 = v;
      c1 = c;
    }
  }
  const int wm1 = wave_max_dpp(m1);
  const int wc1 = wave_min_dpp(m1 == wm1 ? c1 : INT_MAX);
  int m2 = INT_MIN;
  for (int c = lane; c < per_class; c += kWave) m2 = max(m2, c != wc1 ? mc[c] : INT_MIN);
  const int wm2 = wave_max_dpp(m2);
  for (int e0 = 0; e0 < E; e0 += kWave) {
    const int e = e0 + lane;
    const int cell = ccand[min(e, E - 1)];
    const bool mine = e < E && cell >= 0 && cell < N && cell / per_class == i;
    // the reads use a valid cell of class i for every candidate (so they
    // are unconditional and overlap); other candidates' values are unused
    const int local = mine ? cell - i * per_class : 0;
    const int ti = local / B;
    const int t = c_tp[ti], first = c_optoff[ti];
    const int lo = crlo[local], hi = crhi[local];
    const uint8_t rev = mrow[i * per_class + local];
    const int nr = hi >= lo ? hi - lo + 1 : 0;
    // M at rlo, the same value as the option's (every lane takes part in
    // the lookup)
    const int m_lo = min(__builtin_amdgcn_ds_bpermute(4 * max(G - t * (nr > 0 ? lo : 1), 0), hreg),
                         __float_as_int(1.0f));
    if (!mine) continue;
    TileInfo *tl = tiles + (size_t)o * E + e;
    const int u = max(0, local == wc1 ? wm2 : wm1);
    if (R == 0) {
      tl->cls = i; tl->t = t; tl->cell = cell;
      tl->rlo = nr > 0 ? lo : 1;
      tl->rhi = nr > 0 ? hi : 0;
      tl->state = rev ? 1 : 0;
      tl->toff = i * PPc + first + (nr > 0 ? lo : 1) - 1;
      tl->u_m = u;
      tl->m_m = nr > 0 ? m_lo : 0;
    } else {
      tl->u_p = u;
      tl->m_p = nr > 0 ? m_lo : 0;
    }
  }
  if (i == 0 && lane == 0) base[o * 2 + R] = max(0, wm1);  // 0: the empty allocation
}

// Sampled ratio of r replicas: min(1, fl32(fl32(r * c) / lambda)) as bits.
__device__ __forceinline__ int sampled_ratio(float rf, float cs, double rcp) {
  const float capacity = rf * cs;
  return __float_as_int(fminf((float)((double)capacity * rcp), 1.0f));
}

// The same quotient without the clamp at 1, for use as min(q, M) with M <= 1
// (the clamp cannot change that minimum).
__device__ __forceinline__ int sampled_quotient(float rf, float cs, double rcp) {
  const float capacity = rf * cs;
  return __float_as_int((float)((double)capacity * rcp));
}

// Pairwise sum (balanced tree over the sample order, zero-padded to a power
// of two) of n copies of c.  Every full aligned block of 2^j copies sums to
// 2^j c exactly, so the tree is its lowest set bit of n as one full block,
// then one addition per higher set bit, innermost first.
__device__ __forceinline__ double pairwise_run(double c, int64_t n) {
  if (n <= 0) return 0.0;
  int64_t low = n & -n;
  double acc = (double)low * c;
  for (int64_t rest = n - low; rest != 0; rest -= low) {
    low = rest & -rest;
    acc = (double)low * c + acc;
  }
  return acc;
}

// Largest replica range handled by the unrolled scan; longer ranges use the
// crossing search.
constexpr int kScanMax = 4;

// Default grid of the exclusion scorer: three wavefronts per SIMD (1024
// SIMDs).  On the 4-class, G = 64 workload (about 7,100 items) three per
// SIMD ran the scorer in 9.0-9.1 us against 9.5 us with four, 10.0 with 2.5
// and 10.7-11.2 with two.
constexpr int kScorerWaves = 3072;

// Samples of one chunk.  VEC (S a multiple of 4): each group of 4 samples
// of a lane lies wholly below S or wholly past it; every group is fetched by
// one 16-byte load at an in-bounds address (a group past S reads the tile's
// last 4 samples, values that are never used), so the loads are unconditional
// and the compiler's wait counts stay exact.  Otherwise single loads,
// predicated per sample.
template <int SPL, bool VEC>
__device__ __forceinline__ void load_chunk(const float *__restrict__ cap_s, const float *__restrict__ tail_s,
                                           size_t tbase, int s_first, int S, bool live, float (&cs)[SPL],
                                           float (&ls)[SPL]) {
  if constexpr (VEC) {
#pragma unroll
    for (int v4 = 0; v4 < SPL / 4; ++v4) {
      const size_t at = tbase + (size_t)min(s_first + 4 * v4, S - 4);
      const float4 c4 = *reinterpret_cast<const float4 *>(cap_s + at);
      const float4 l4 = *reinterpret_cast<const float4 *>(tail_s + at);
      cs[4 * v4 + 0] = c4.x; cs[4 * v4 + 1] = c4.y; cs[4 * v4 + 2] = c4.z; cs[4 * v4 + 3] = c4.w;
      ls[4 * v4 + 0] = l4.x; ls[4 * v4 + 1] = l4.y; ls[4 * v4 + 2] = l4.z; ls[4 * v4 + 3] = l4.w;
    }
  } else {
#pragma unroll
    for (int q = 0; q < SPL; ++q) {
      const bool in = live && s_first + q < S;
      cs[q] = in ? cap_s[tbase + s_first + q] : 0.0f;
      ls[q] = in ? tail_s[tbase + s_first + q] : 0.0f;
    }
  }
}

// Everything one work item reads: its work-list entry, U and M at rlo of
// both realisations (one 16-byte load of the tile record), and -- unless no
// sample can matter (triv) -- the lane's samples and M and the capacity
// threshold of option rlo + min(lane, nr - 1) of both realisations (a scan
// reads M lane by lane, the crossing search looks both up across lanes).
template <int SPL>
struct ScoreItem {
  int4 ent;
  float cs[SPL], ls[SPL];
  int u0, u1, mr0, mr1;
  int vm0, vm1;
  float vt0, vt1;
  bool triv;
};

// Value of lane idx (0 <= idx < 64) of v, per lane.
__device__ __forceinline__ int lane_lookup(int v, int idx) { return __builtin_amdgcn_ds_bpermute(idx << 2, v); }

// Scenarios of the exclusion scorer.  A work item is one chunk of 64 x SPL
// samples of one live tile; items are numbered over the live tiles only, so
// every wavefront gets the same number of items to within one, and the
// chunks of one tile are neighbours.  Each wavefront of the grid takes the
// items it, it + W, it + 2W, ... (W wavefronts) and runs them as a
// three-stage pipeline: while the current item is evaluated, the list entry
// of the third item ahead, the tile-record words of the second (U and M at
// rlo, both realisations) and the samples and the range's M and thresholds
// of the next are in flight.  All of these are vector loads
// at unconditional (clamped) addresses, so each wait covers exactly the item
// it is for; the per-class constants sit in LDS.  Lane l owns samples
// [c * 64 * SPL + l * SPL, + SPL) of the item's tile, and the chunk's sum
// is written as one partial (a node of the pairwise tree over s).
//
// An item whose M over the whole range is at most U in both realisations
// has tau = U in every scenario, whatever its samples (every term
// min(f_r, M_r) is at most M_r): its samples are not read (the item's loads
// go to one line at the start of the arrays, still unconditionally) and its
// partial is the closed-form pairwise sum of the constant gap U+ - U-.
// M falls along a range (M_r = min(H[G - t*r], 1) with H a prefix
// maximum, as signed integers on its bits), so M at the range's first
// count, which the set-up puts in the tile record, is its largest.
//
// Per realisation, tau = max(U, max_r min(f_r, M_r)) with M_r = H[G - t*r].
// Ranges of at most kScanMax replica counts are scanned.  For longer ones:
// f_r is nondecreasing in r and M_r nonincreasing, so min(f_r, M_r) rises
// while f_r < M_r and falls after; with r* the first r where f_r >= M_r --
// the first r whose capacity threshold the sample reaches -- the maximum is
// max(f_{r*-1}, M_{r*}).
template <int SPL, bool VEC, bool DUMP>
__global__ __launch_bounds__(64) void k_score_excl(
    DevProblem P, const TileInfo *__restrict__ tiles, const int32_t *__restrict__ mopt,
    const float *__restrict__ thr, int32_t n_thr, const int4 *__restrict__ list,
    const float *__restrict__ cap_s, const float *__restrict__ tail_s, int32_t O, int32_t E, int32_t S,
    const int32_t *__restrict__ base, double *__restrict__ partial, int32_t n_chunk,
    float *__restrict__ tau_dump) {
  constexpr int CHUNK = 64 * SPL;
  extern __shared__ int lds[];
  const int lane = threadIdx.x;
  const int wv = (int)blockIdx.x;
  // per-class constants in LDS; then, for ranges longer than a wavefront, M
  // and the thresholds of the range
  double *c_rcp = reinterpret_cast<double *>(lds);
  float *c_slo = reinterpret_cast<float *>(c_rcp + P.K);
  int *Mlds = reinterpret_cast<int *>(c_slo + P.K);
  for (int k = lane; k < P.K; k += kWave) {
    c_rcp[k] = P.rcp_demand[k];
    c_slo[k] = P.slo[k];
  }
  wave_lds_fence();
  // An opaque zero added to every address below: the loads stay vector
  // loads.  (Scalar loads complete out of order, so a wait for any LDS
  // result would also wait for every scalar load in flight, including the
  // next item's.)
  int vz;
  asm volatile("v_mov_b32 %0, 0" : "=v"(vz));
  const int W = (int)gridDim.x;
  // Item it = j * n_chunk + c: chunk c of the tile in place j of the work
  // list (every order's live tiles, longest replica range first).  Items go
  // to the wavefronts in serpentine order: wavefront w takes items w,
  // 2W - 1 - w, 2W + w, 4W - 1 - w, ..., so the wavefronts with the
  // heaviest first items get the lightest second ones.  Positions carry the
  // parity of their round; the two steps are kept as (places, chunks).
  struct Pos { int64_t j; int c; int odd; };
  const int64_t n_list = (int64_t)O * E;
  const int64_t d_even = 2 * (int64_t)W - 1 - 2 * wv, d_odd = 2 * (int64_t)wv + 1;
  const int64_t sj0 = d_even / n_chunk, sj1 = d_odd / n_chunk;
  const int sc0 = (int)(d_even - sj0 * n_chunk), sc1 = (int)(d_odd - sj1 * n_chunk);
  auto advance = [&](Pos q) {
    q.j += q.odd ? sj1 : sj0;
    q.c += q.odd ? sc1 : sc0;
    if (q.c >= n_chunk) { q.c -= n_chunk; ++q.j; }
    q.odd ^= 1;
    return q;
  };
  auto uniform4 = [](int4 v) {
    return make_int4(__builtin_amdgcn_readfirstlane(v.x), __builtin_amdgcn_readfirstlane(v.y),
                     __builtin_amdgcn_readfirstlane(v.z), __builtin_amdgcn_readfirstlane(v.w));
  };
  auto list_at = [&](const Pos &p) { return list[(p.j < n_list ? p.j : 0) + vz]; };
  // Issues the tile-record load of an item whose list entry is known.
  // Items without a tile read the first record instead.
  auto issue_head = [&](ScoreItem<SPL> &X) {
    const int4 en = X.ent;
    const bool live = en.x >= 0;
    const int o = en.w >> 8;
    const size_t tile = live ? (size_t)o * E + en.x : 0;
    const int4 h = *reinterpret_cast<const int4 *>(&tiles[tile + vz].u_m);  // (u_m, u_p, m_m, m_p)
    X.u0 = h.x;
    X.u1 = h.y;
    X.mr0 = h.z;
    X.mr1 = h.w;
  };
  // Decides, from an item's record, whether its samples can matter, and
  // issues their loads and the range's M and thresholds if so.  The test
  // uses the comparisons the evaluation makes (signed integers on binary32
  // bits).
  auto issue_samples = [&](ScoreItem<SPL> &X, const Pos &p) {
    const int4 en = X.ent;
    const int nr = en.z >> 16, o = en.w >> 8;
    const int m0 = __builtin_amdgcn_readfirstlane(X.mr0), m1 = __builtin_amdgcn_readfirstlane(X.mr1);
    const int u0 = __builtin_amdgcn_readfirstlane(X.u0), u1 = __builtin_amdgcn_readfirstlane(X.u1);
    const bool triv = !DUMP && en.x >= 0 && m0 <= u0 && m1 <= u1;
    X.triv = triv;
    const bool live = en.x >= 0 && !triv;
    const size_t tile = live ? (size_t)o * E + en.x : 0;
    load_chunk<SPL, VEC>(cap_s, tail_s, tile * S, live ? p.c * CHUNK + lane * SPL : 0, S, live, X.cs, X.ls);
    const size_t row0 = live ? (size_t)o * 2 * n_thr : 0, row1 = live ? row0 + n_thr : 0;
    const int at = (live ? en.y : 0) + (live && nr > 0 ? min(lane, nr - 1) : 0) + vz;
    X.vm0 = mopt[row0 + at];
    X.vm1 = mopt[row1 + at];
    X.vt0 = thr[row0 + at];
    X.vt1 = thr[row1 + at];
  };
  // Evaluates an item whose loads were issued.
  auto evaluate = [&](const ScoreItem<SPL> &X, const Pos &p) {
    const int4 en = X.ent;
    if (en.x < 0) return;  // no tile (uniform)
    const int e = en.x, toff = en.y, rlo = en.z & 0xFFFF, nr = en.z >> 16;
    const int cls = en.w & 0x3F, state = (en.w >> 6) & 3, o = en.w >> 8;
    const size_t tile = (size_t)o * E + e;
    const int s_first = p.c * CHUNK + lane * SPL;
    if (X.triv) {
      // the chunk's samples past S add 0
      if (lane == 0) {
        const int u0 = __builtin_amdgcn_readfirstlane(X.u0), u1 = __builtin_amdgcn_readfirstlane(X.u1);
        const int n = min(CHUNK, S - p.c * CHUNK);
        partial[tile * n_chunk + p.c] =
            pairwise_run((double)__int_as_float(u1) - (double)__int_as_float(u0), n);
      }
      return;
    }
    if (DUMP && (state != 0 || nr == 0)) {
      // listed only when dumping: a revealed cell keeps the base values; a
      // cell no replica count reaches leaves tau at U
      const int vm = state != 0 ? base[o * 2 + 0] : X.u0;
      const int vp = state != 0 ? base[o * 2 + 1] : X.u1;
      for (int q = 0; q < SPL; ++q) {
        if (s_first + q < S) {
          tau_dump[(tile * S + s_first + q) * 2 + 0] = __int_as_float(vm);
          tau_dump[(tile * S + s_first + q) * 2 + 1] = __int_as_float(vp);
        }
      }
      return;
    }
    const double rcp = c_rcp[cls];
    const float slo = c_slo[cls];
    // tau = max(U, best over the range): U (uniform, in scalar registers)
    // enters the accumulators with their first update -- every path below
    // writes each accumulator (a listed tile has nr >= 1).  A sampled tail
    // above the SLO makes every option on the cell worth 0, leaving tau = U:
    // the sample's capacity is taken as 0 instead, whose ratios (0) and
    // crossings (M <= 0 where reached) cannot raise tau above U >= 0.
    const int u0 = __builtin_amdgcn_readfirstlane(X.u0), u1 = __builtin_amdgcn_readfirstlane(X.u1);
    int am[SPL], ap[SPL];
    float cs[SPL];
#pragma unroll
    for (int q = 0; q < SPL; ++q) cs[q] = X.ls[q] <= slo ? X.cs[q] : 0.0f;
    if (nr <= kScanMax) {
      // pairs of replica counts, then a single one when nr is odd
#pragma unroll
      for (int j = 0; j < kScanMax; j += 2) {
        if (j + 1 < nr) {
          // M <= 1 lets min(f, M) use the unclamped quotient
          const int mm0 = __builtin_amdgcn_readlane(X.vm0, j), mp0 = __builtin_amdgcn_readlane(X.vm1, j);
          const int mm1 = __builtin_amdgcn_readlane(X.vm0, j + 1);
          const int mp1 = __builtin_amdgcn_readlane(X.vm1, j + 1);
          const float r1 = (float)(rlo + j), r2 = (float)(rlo + j + 1);
#pragma unroll
          for (int q = 0; q < SPL; ++q) {
            const int f1 = sampled_quotient(r1, cs[q], rcp);
            const int f2 = sampled_quotient(r2, cs[q], rcp);
            am[q] = max(j == 0 ? u0 : am[q], max(min(f1, mm0), min(f2, mm1)));
            ap[q] = max(j == 0 ? u1 : ap[q], max(min(f1, mp0), min(f2, mp1)));
          }
        } else if (j < nr) {
          const int mm0 = __builtin_amdgcn_readlane(X.vm0, j), mp0 = __builtin_amdgcn_readlane(X.vm1, j);
          const float r1 = (float)(rlo + j);
#pragma unroll
          for (int q = 0; q < SPL; ++q) {
            const int f1 = sampled_quotient(r1, cs[q], rcp);
            am[q] = max(j == 0 ? u0 : am[q], min(f1, mm0));
            ap[q] = max(j == 0 ? u1 : ap[q], min(f1, mp0));
          }
        }
      }
    } else {
      // All 2 x SPL searches advance together.  pos counts the leading
      // thresholds the sample does not reach (NaN is never reached); the
      // predicate is monotone in the option, so after the steps
      // 2^(steps-1), ..., 1 pos is the first crossing.
      int steps = 0;
      while ((1 << steps) <= nr) ++steps;  // ceil(log2(nr + 1))
      if (nr < kWave) {
        // Option rlo + j of the range sits in lane j.  The lanes past the
        // range hold a threshold every sample reaches (-inf) and no option
        // (M = INT_MIN), so the search never passes nr and needs no index
        // clamp: a lookup index stays below 2^steps - 1 <= 63.  pos is kept
        // in bytes (4 pos), the lane address of the lookups.  Lane j of rb
        // holds the replica count below option j (0 for j = 0: its ratio,
        // 0, cannot raise tau).  Each step issues all 2 x SPL cross-lane
        // lookups before the first compare (the scheduling barriers keep
        // them together, so their latencies overlap).
        const bool in_range = lane < nr;
        const int t0 = in_range ? __float_as_int(X.vt0) : (int)0xFF800000u;
        const int t1 = in_range ? __float_as_int(X.vt1) : (int)0xFF800000u;
        const int m0 = in_range ? X.vm0 : INT_MIN;
        const int m1 = in_range ? X.vm1 : INT_MIN;
        const int rb = __float_as_int(lane == 0 ? 0.0f : (float)(rlo + lane - 1));
        // the first step probes one lane for every search (pos = 0): a
        // uniform threshold, read into a scalar register
        const int stp0 = 1 << (steps - 1);
        const float f0m = __int_as_float(__builtin_amdgcn_readlane(t0, stp0 - 1));
        const float f0p = __int_as_float(__builtin_amdgcn_readlane(t1, stp0 - 1));
        int pb[SPL][2];
#pragma unroll
        for (int q = 0; q < SPL; ++q) {
          pb[q][0] = !(cs[q] >= f0m) ? 4 * stp0 : 0;
          pb[q][1] = !(cs[q] >= f0p) ? 4 * stp0 : 0;
        }
        for (int stp = stp0 >> 1; stp > 0; stp >>= 1) {
          const int off = 4 * (stp - 1);
          int th[SPL][2];
#pragma unroll
          for (int q = 0; q < SPL; ++q) {
            th[q][0] = __builtin_amdgcn_ds_bpermute(pb[q][0] + off, t0);
            th[q][1] = __builtin_amdgcn_ds_bpermute(pb[q][1] + off, t1);
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int q = 0; q < SPL; ++q) {
#pragma unroll
            for (int side = 0; side < 2; ++side)
              pb[q][side] += !(cs[q] >= __int_as_float(th[q][side])) ? 4 * stp : 0;
          }
        }
        // tau candidate: max(f of the replica count below the crossing,
        // M at the crossing).  Below the crossing f < M <= 1, so the
        // unclamped quotient is the ratio.
        int mj[SPL][2], rj[SPL][2];
#pragma unroll
        for (int q = 0; q < SPL; ++q) {
          mj[q][0] = __builtin_amdgcn_ds_bpermute(pb[q][0], m0);
          mj[q][1] = __builtin_amdgcn_ds_bpermute(pb[q][1], m1);
          rj[q][0] = __builtin_amdgcn_ds_bpermute(pb[q][0], rb);
          rj[q][1] = __builtin_amdgcn_ds_bpermute(pb[q][1], rb);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < SPL; ++q) {
          const int fm = sampled_quotient(__int_as_float(rj[q][0]), cs[q], rcp);
          const int fp = sampled_quotient(__int_as_float(rj[q][1]), cs[q], rcp);
          am[q] = max(u0, max(fm, mj[q][0]));
          ap[q] = max(u1, max(fp, mj[q][1]));
        }
      } else {
        // a range of a wavefront's length or more: M and the thresholds go
        // to LDS
        int pos[SPL][2];
#pragma unroll
        for (int q = 0; q < SPL; ++q) pos[q][0] = pos[q][1] = 0;
        const int32_t *Mm = mopt + (size_t)o * 2 * n_thr + toff, *Mp = Mm + n_thr;
        const float *Tm = thr + (size_t)o * 2 * n_thr + toff, *Tp = Tm + n_thr;
        float *Tl = reinterpret_cast<float *>(Mlds + 2 * nr);
        wave_lds_fence();  // the previous item's reads of this LDS are done
        for (int j = lane; j < nr; j += kWave) {
          Mlds[j] = Mm[j];
          Mlds[nr + j] = Mp[j];
          Tl[j] = Tm[j];
          Tl[nr + j] = Tp[j];
        }
        wave_lds_fence();
        for (int stp = 1 << (steps - 1); stp > 0; stp >>= 1) {
          float th[SPL][2];
#pragma unroll
          for (int q = 0; q < SPL; ++q) {
            th[q][0] = Tl[min(pos[q][0] + stp - 1, nr - 1)];
            th[q][1] = Tl[nr + min(pos[q][1] + stp - 1, nr - 1)];
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int q = 0; q < SPL; ++q) {
#pragma unroll
            for (int side = 0; side < 2; ++side) {
              const int idx = pos[q][side] + stp - 1;
              const bool below = !(cs[q] >= th[q][side]);
              pos[q][side] += (idx < nr && below) ? stp : 0;
            }
          }
        }
        int mj[SPL][2];
#pragma unroll
        for (int q = 0; q < SPL; ++q) {
          mj[q][0] = Mlds[min(pos[q][0], nr - 1)];
          mj[q][1] = Mlds[nr + min(pos[q][1], nr - 1)];
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < SPL; ++q) {
#pragma unroll
          for (int side = 0; side < 2; ++side) {
            const int j = pos[q][side];
            const int fprev = sampled_ratio((float)(rlo + j - 1), cs[q], rcp);
            const int v = max(j > 0 ? fprev : INT_MIN, j < nr ? mj[q][side] : INT_MIN);
            if (side == 0) am[q] = max(u0, v);
            else ap[q] = max(u1, v);
          }
        }
      }
    }
    double gq[SPL];
    // samples past S add 0 (the chunk holds none of them unless it is the
    // tile's last and S is not a multiple of its size)
    const bool full = (p.c + 1) * CHUNK <= S;
    if (full) {
#pragma unroll
      for (int q = 0; q < SPL; ++q) {
        const int tm = am[q], tp = ap[q];
        gq[q] = (double)__int_as_float(tp) - (double)__int_as_float(tm);
        if (DUMP) {
          tau_dump[(tile * S + s_first + q) * 2 + 0] = __int_as_float(tm);
          tau_dump[(tile * S + s_first + q) * 2 + 1] = __int_as_float(tp);
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < SPL; ++q) {
        const int tm = am[q], tp = ap[q];
        const bool live = s_first + q < S;
        gq[q] = live ? (double)__int_as_float(tp) - (double)__int_as_float(tm) : 0.0;
        if (DUMP && live) {
          tau_dump[(tile * S + s_first + q) * 2 + 0] = __int_as_float(tm);
          tau_dump[(tile * S + s_first + q) * 2 + 1] = __int_as_float(tp);
        }
      }
    }
    // pairwise tree: within the lane's SPL consecutive samples, then lanes
#pragma unroll
    for (int w = 1; w < SPL; w <<= 1) {
#pragma unroll
      for (int j = 0; j + w < SPL; j += 2 * w) gq[j] = gq[j] + gq[j + w];
    }
    const double v = wave_pairwise_sum(gq[0]);
    if (lane == 0) partial[tile * n_chunk + p.c] = v;
  };

  // Items a (current), m (next) and n (second next).
  Pos pa;
  pa.j = wv / n_chunk;
  pa.c = wv - (int)pa.j * n_chunk;
  pa.odd = 0;
  ScoreItem<SPL> A, B, C;
  // the first three list entries are requested together
  const int4 raw_a = list_at(pa);
  Pos pm = advance(pa);
  const int4 raw_m = list_at(pm);
  Pos pn = advance(pm);
  int4 raw_n = list_at(pn);
  A.ent = uniform4(raw_a);
  if (pa.j >= n_list) A.ent.x = -1;
  issue_head(A);
  B.ent = uniform4(raw_m);
  if (pm.j >= n_list) B.ent.x = -1;
  issue_head(B);
  issue_samples(A, pa);
  // One pipeline stage: the list entry of the third item ahead and the
  // constants of the second are requested, the next item's samples are
  // issued (its constants arrived during the previous stage), the current
  // item is evaluated.  The three item buffers rotate roles (no copies, so
  // no early waits).  Places only grow, so the first end marker ends the
  // wavefront's work.
  auto stage = [&](ScoreItem<SPL> &cur, ScoreItem<SPL> &mid, ScoreItem<SPL> &nxt) {
    nxt.ent = uniform4(raw_n);
    if (pn.j >= n_list) nxt.ent.x = -1;
    const Pos pq = advance(pn);
    const int4 raw_q = list_at(pq);
    issue_head(nxt);
    issue_samples(mid, pm);
    evaluate(cur, pa);
    pa = pm;
    pm = pn;
    pn = pq;
    raw_n = raw_q;
  };
  for (;;) {
    if (A.ent.x < 0) break;
    stage(A, B, C);
    if (B.ent.x < 0) break;
    stage(B, C, A);
    if (C.ent.x < 0) break;
    stage(C, A, B);
  }
}

// Tile score of the exclusion scorer: Gamma_t - (sum over s of the
// scenario's gap) / S.  A tile with no replica count on its cell has the
// same gap u_p - u_m in every scenario and was not visited by the scorer.
__device__ __forceinline__ bool excl_constant_tile(const TileInfo &tl) { return tl.rhi < tl.rlo; }

__device__ __forceinline__ double excl_constant_sum(const TileInfo &tl, int32_t S) {
  return pairwise_run((double)__int_as_float(tl.u_p) - (double)__int_as_float(tl.u_m), S);
}

// Order-preserving key of a score: a larger score has a larger key, and
// -0.0 counts as +0.0 (scores compare equal there).  Every number's key is
// above 0, which stands for "no candidate".
__device__ __forceinline__ uint64_t score_key(double x) {
  const uint64_t b = (uint64_t)__double_as_longlong(x + 0.0);
  return (b >> 63) ? ~b : (b | (1ull << 63));
}

// Tie-break key among equal scores (smaller wins): TP degree, then cell,
// then candidate index (TP <= 4096 and cells < 2^16 by the problem limits).
__device__ __forceinline__ uint64_t tie_key(int tp, int cell, int e) {
  return ((uint64_t)(uint32_t)tp << 48) | ((uint64_t)(uint32_t)cell << 32) | (uint64_t)(uint32_t)e;
}

template <int kCtrl>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)v, kCtrl, 0xF, 0xF, true);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(v >> 32), kCtrl, 0xF, 0xF, true);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// Maximum (kMax) or minimum of a 64-bit key over the 64 lanes, by the same
// DPP pattern as wave_max_dpp.  Wave-uniform result; every lane active.
template <bool kMax>
__device__ __forceinline__ uint64_t wave_ext_u64(uint64_t v) {
  auto pick = [](uint64_t a, uint64_t b) { return kMax ? (a > b ? a : b) : (a < b ? a : b); };
  v = pick(v, dpp_u64<0xB1>(v));
  v = pick(v, dpp_u64<0x4E>(v));
  v = pick(v, dpp_u64<0x141>(v));
  v = pick(v, dpp_u64<0x140>(v));
  return pick(pick(readlane_u64(v, 0), readlane_u64(v, 16)), pick(readlane_u64(v, 32), readlane_u64(v, 48)));
}

// Scores and best candidate of the exclusion scorer: one block per order
// of one wavefront per 128 candidates (at most 16), lane l of wavefront w
// taking candidates 128 w + l, 128 w + l + 64, then the next 128 nw, ...
// two at a time (their loads overlap).  Each tile's partials (at most 16
// here) are summed by the pairwise tree in registers.  The arg-max is two
// key reductions per wavefront -- the largest score, then the smallest
// (TP, cell, index) among the lanes holding it, the order that `better`
// defines -- then the same over the wavefronts' results.
constexpr int kFinalizeMaxWaves = 16;

__global__ __launch_bounds__(64 * kFinalizeMaxWaves) void k_finalize_excl(
    const TileInfo *__restrict__ tiles, int32_t E, int32_t S, const int32_t *__restrict__ base,
    const double *__restrict__ partial, int64_t n_partial, double *__restrict__ score,
    double *__restrict__ gap_now, int32_t *__restrict__ best) {
  __shared__ uint64_t s_key[kFinalizeMaxWaves], s_tie[kFinalizeMaxWaves];
  const int o = blockIdx.x, lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const double gap = (double)__int_as_float(base[o * 2 + 1]) - (double)__int_as_float(base[o * 2 + 0]);
  int p2 = 1;
  while (p2 < n_partial) p2 <<= 1;
  uint64_t kbest = 0, tbest = ~0ull;
  for (int e0 = wave * 2 * kWave + lane; e0 < E; e0 += nw * 2 * kWave) {
    double v[2][16];
    TileInfo tl[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      // the partials are read together with the tile record (entries of
      // tiles the scorer did not visit are not used)
      const int e = e0 + u * kWave;
      const size_t tile = (size_t)o * E + (e < E ? e : 0);
      const double *x = partial + tile * n_partial;
#pragma unroll
      for (int j = 0; j < 16; ++j) v[u][j] = j < n_partial ? x[j] : 0.0;
      tl[u] = tiles[tile];
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int e = e0 + u * kWave;
      if (e >= E) continue;
      double sc = 0.0;  // a revealed cell: nothing to learn
      if (tl[u].state < 0) {
        sc = __builtin_nan("");
      } else if (tl[u].state == 0) {
        double sum;
        if (excl_constant_tile(tl[u])) {
          sum = excl_constant_sum(tl[u], S);
        } else {
#pragma unroll
          for (int w = 1; w < 16; w <<= 1) {
            if (w < p2) {
#pragma unroll
              for (int j = 0; j + w < 16; j += 2 * w) v[u][j] = v[u][j] + v[u][j + w];
            }
          }
          sum = v[u][0];
        }
        sc = gap - sum / (double)S;
        const uint64_t k = score_key(sc), t = tie_key(tl[u].t, tl[u].cell, e);
        if (k > kbest || (k == kbest && t < tbest)) {
          kbest = k;
          tbest = t;
        }
      }
      score[(size_t)o * E + e] = sc;
    }
  }
  const uint64_t kmax = wave_ext_u64<true>(kbest);
  const uint64_t tmin = wave_ext_u64<false>(kbest == kmax ? tbest : ~0ull);
  if (lane == 0) {
    s_key[wave] = kmax;
    s_tie[wave] = tmin;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t K = 0, T = ~0ull;
    for (int w = 0; w < nw; ++w) {
      if (s_key[w] > K || (s_key[w] == K && s_tie[w] < T)) {
        K = s_key[w];
        T = s_tie[w];
      }
    }
    if (best) best[o] = K != 0 ? (int32_t)(uint32_t)T : -1;
    if (gap_now) gap_now[o] = gap;
  }
}

// Scores and best candidate, many partials per tile: one wavefront per
// candidate sums the tile's partials; then a second pass picks the best.
__global__ __launch_bounds__(256) void k_tile_scores_wave(const TileInfo *__restrict__ tiles, int32_t E,
                                                          int32_t S, const int32_t *__restrict__ base,
                                                          const double *__restrict__ partial,
                                                          int64_t n_partial, double *__restrict__ score) {
  const int o = blockIdx.y;
  const int e = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (e >= E) return;
  const size_t tile = (size_t)o * E + e;
  const TileInfo tl = tiles[tile];
  double sc = 0.0;
  if (tl.state < 0) sc = __builtin_nan("");
  if (tl.state == 0) {
    const double gap = (double)__int_as_float(base[o * 2 + 1]) - (double)__int_as_float(base[o * 2 + 0]);
    const double sum = excl_constant_tile(tl) ? excl_constant_sum(tl, S)
                                              : wave_tree_sum(partial + tile * n_partial, n_partial);
    sc = gap - sum / (double)S;
  }
  if ((threadIdx.x & 63) == 0) score[tile] = sc;
}

__global__ __launch_bounds__(256) void k_pick_best(const TileInfo *__restrict__ tiles, int32_t E,
                                                   const int32_t *__restrict__ base,
                                                   const double *__restrict__ score,
                                                   double *__restrict__ gap_now, int32_t *__restrict__ best) {
  __shared__ Pick s_pick[4];
  const int o = blockIdx.x;
  Pick mine{0.0, 0, 0, -1};
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    const TileInfo tl = tiles[(size_t)o * E + e];
    if (tl.state != 0) continue;
    const Pick c{score[(size_t)o * E + e], tl.t, tl.cell, e};
    if (better(c, mine)) mine = c;
  }
  mine = wave_best(mine);
  if ((threadIdx.x & 63) == 0) s_pick[threadIdx.x >> 6] = mine;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w)
      if (better(s_pick[w], mine)) mine = s_pick[w];
    if (best) best[o] = mine.e;
    if (gap_now)
      gap_now[o] = (double)__int_as_float(base[o * 2 + 1]) - (double)__int_as_float(base[o * 2 + 0]);
  }
}

// ---------------------------------------------------------------------------
// Finalize: score = Gamma_t - (pairwise sum of partials) / S, and the argmax.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_finalize(DevProblem P, const CandInfo *__restrict__ info,
                                                 const uint8_t *__restrict__ measured, int32_t E,
                                                 int32_t S, const int32_t *__restrict__ base,
                                                 const double *__restrict__ partial,
                                                 int64_t n_partial, double *__restrict__ score,
                                                 double *__restrict__ gap_now,
                                                 int32_t *__restrict__ best) {
  const int o = blockIdx.x, lane = threadIdx.x;
  const double gap = (double)__int_as_float(base[o * 2 + 1]) - (double)__int_as_float(base[o * 2 + 0]);
  if (lane == 0 && gap_now) gap_now[o] = gap;
  Pick mine{0.0, 0, 0, -1};
  for (int e = lane; e < E; e += kWave) {
    const CandInfo ci = info[e];
    const size_t tile = (size_t)o * E + e;
    if (ci.cls < 0) {
      score[tile] = __builtin_nan("");
      continue;
    }
    if (measured[(size_t)o * P.N + ci.cell]) {
      score[tile] = 0.0;
      continue;
    }
    // pairwise tree over the partials, zero-padded to a power of two; the
    // padding adds exact zeros, so the open stack folds from the top
    const double *x = partial + tile * n_partial;
    double stack[32];
    int depth = 0;
    for (int64_t i = 0; i < n_partial; ++i) {
      double v = x[i];
      for (int64_t m = i; m & 1; m >>= 1) v = stack[--depth] + v;
      stack[depth++] = v;
    }
    double sum = stack[depth - 1];
    for (int d = depth - 2; d >= 0; --d) sum = stack[d] + sum;
    const double sc = gap - sum / (double)S;
    score[tile] = sc;
    const Pick cand{sc, ci.tp, ci.cell, e};
    if (better(cand, mine)) mine = cand;
  }
  mine = wave_best(mine);
  if (lane == 0 && best) best[o] = mine.e;
}

// ---------------------------------------------------------------------------
// Certificate: one wavefront per order.
// ---------------------------------------------------------------------------
// State of one order (Section 4.2) given both allocations and whether the
// gap is within eps: 2 when a class is critical and even the optimistic
// allocation misses a floor; 1 when the conservative allocation meets the
// floors, every cell it commits to is measured with its tail upper bound
// within the SLO, and the gap is within eps; 0 otherwise.
__device__ __forceinline__ int certificate_state(const DevProblem &P, const int8_t *__restrict__ bmap,
                                                 const uint8_t *__restrict__ measured,
                                                 const float *__restrict__ tail_hi, size_t off, int fm_m,
                                                 int fm_p, const int *tm_index, const int *tm_rep,
                                                 bool gap_ok) {
  if (P.has_floor && !fm_p) return 2;
  bool ok = fm_m != 0;
  for (int k = 0; k < P.K && ok; ++k) {
    const int r = tm_rep[k];
    if (r == 0) continue;
    const int cell = cell_of(P, k, tm_index[k], bmap[k * (P.G + 1) + r]);
    if (!measured[off + cell]) ok = false;
    else if (!(tail_hi[off + cell] <= P.slo[k])) ok = false;
  }
  return (ok && gap_ok) ? 1 : 0;
}

// Result of one realisation's solve in a certificate: tau, floors, goodput
// (binary32 and, under the whole objective, level (3)'s binary64 total) and
// the allocation.
struct CertRec {
  int32_t tau, floors_met;
  float goodput;
  int32_t pad;
  double goodput64;
  int32_t tp_index[kMaxClasses], replicas[kMaxClasses];
};

__device__ __forceinline__ void write_cert_rec(CertRec *me, int K, int tau, int fm, float gp, double g64,
                                               const WaveAlloc &wa) {
  const int lane = threadIdx.x & (kWave - 1);
  if (lane == 0) {
    me->tau = tau;
    me->floors_met = fm;
    me->goodput = gp;
    me->goodput64 = g64;
  }
  for (int k = lane; k < K; k += kWave) {
    me->tp_index[k] = wa.tp_index[k];
    me->replicas[k] = wa.replicas[k];
  }
}

// Certificate (Section 4.2): block (R, o) solves realisation R of order o
// (0: conservative, 1: optimistic) and keeps its result in a record;
// k_certify_state then forms each order's gap and state from the two.
// STAGE: inputs staged in LDS (1) or read from global memory (0), fixed at
// compile time so that every access compiles for its own memory.
template <int STAGE>
__global__ __launch_bounds__(64) void k_certify(DevProblem P, const int8_t *__restrict__ bmap,
                                                const float *__restrict__ cap_lo,
                                                const float *__restrict__ cap_hi,
                                                const float *__restrict__ tail_lo,
                                                const float *__restrict__ tail_hi, AllocOut cons, AllocOut opt,
                                                CertRec *__restrict__ rec) {
  constexpr int stage = STAGE;
  extern __shared__ int lds[];
  const int R = blockIdx.x, o = blockIdx.y;
  const size_t off = (size_t)o * P.N;
  int *t_index = lds + 3 * (P.G + 1);
  int *t_rep = t_index + kMaxClasses;
  WaveAlloc wa{t_index, t_rep};
  const StageArea A = stage_area(P, t_rep + kMaxClasses);
  const int8_t *bm = bmap;
  Realisation rz = R == 0 ? Realisation{cap_lo + off, tail_hi + off, -1, 0.0f, 0.0f}
                          : Realisation{cap_hi + off, tail_lo + off, -1, 0.0f, 0.0f};
  if (stage) {
    stage_copy_bmap(P, bmap, A.bmap);
    stage_copy_cells(P, rz.cap, rz.tail, A.cap, A.tail);
    bm = A.bmap;
    rz = Realisation{A.cap, A.tail, -1, 0.0f, 0.0f};
    __syncthreads();
  }
  int fm;
  float gp;
  const int tau = wave_solve(P, bm, rz, lds, &fm, &wa, &gp);
  write_alloc(R == 0 ? cons : opt, o, P.K, tau, fm, gp, wa);
  write_cert_rec(rec + (size_t)o * 2 + R, P.K, tau, fm, gp, 0.0, wa);
}

// Gap and state of each order from its two records: the max-min gap
// tau+ - tau-, and with lex the goodput gap |gp+ - gp-| / max(gp+, gp-) (0
// when both are 0) of level (3)'s totals; within eps means every stage is.
__global__ __launch_bounds__(64) void k_certify_state(DevProblem P, const int8_t *__restrict__ bmap,
                                                      const float *__restrict__ tail_hi,
                                                      const uint8_t *__restrict__ measured, float eps,
                                                      const CertRec *__restrict__ rec, int lex,
                                                      int32_t *__restrict__ state, double *__restrict__ gap_mm_out,
                                                      double *__restrict__ gap_gp_out) {
  const int o = blockIdx.x;
  if (threadIdx.x != 0) return;
  const size_t off = (size_t)o * P.N;
  const CertRec *m = rec + (size_t)o * 2, *p = m + 1;
  const double gap_mm = (double)__int_as_float(p->tau) - (double)__int_as_float(m->tau);
  bool ok = gap_mm <= (double)eps;
  if (gap_mm_out) gap_mm_out[o] = gap_mm;
  if (lex) {
    const double g64_m = m->goodput64, g64_p = p->goodput64;
    const double top = g64_p > g64_m ? g64_p : g64_m;
    const double gap_gp = top > 0.0 ? fabs(g64_p - g64_m) / top : 0.0;
    if (gap_gp_out) gap_gp_out[o] = gap_gp;
    ok = ok && gap_gp <= (double)eps;
  }
  state[o] = certificate_state(P, bmap, measured, tail_hi, off, m->floors_met, p->floors_met, m->tp_index,
                               m->replicas, ok);
}

// ---------------------------------------------------------------------------
// The whole lexicographic objective (Section 3): after levels (1) floors and
// (2) max-min fulfillment, (3) the largest served goodput over allocations
// that keep every ratio at least tau* (and the floors), then (4) the fewest
// GPUs; remaining ties go to the smallest (TP, replicas) of each class in
// class order, empty first.  Served goodput of an option is min(lambda,
// fl32(r c)) when its tail is within the SLO, else 0; totals are binary64
// sums taken from the last class to the first:
//   V_K[g] = (0, 0 GPUs);  V_k[g] = best over allowed options o of class k
//   with cost <= g of (served_o + V_{k+1}[g - cost], cost + GPUs of it),
// best = larger goodput, then fewer GPUs, then the earlier option.  One
// wavefront.  Options of one cost reach the same budgets with the same
// completion, so each class first merges its allowed options per cost c into
// the largest served rate (the earliest option among equal ones) -- no other
// option of that cost can be the best at any budget -- and the layer update
// runs over costs, lanes over the budgets g:
//   V_k[g] = best of (V_{k+1}[g] if empty allowed) and, for c = 1..g,
//            (A_k[c] + V_{k+1}[g - c], c + GPUs of it),
// equal (goodput, GPUs) going to the earlier option (the empty one first).
// The choice of every (class, budget) is kept, and the allocation is read
// in class order from the full budget.
// ---------------------------------------------------------------------------
// A budget's entry of the layer: its best goodput (-inf: no allowed
// completion) and key = GPUs << 16 (the low 16 bits zero).
struct alignas(16) LexCell {
  double gp;
  int key;
  int pad;
};

struct LexLds {
  LexCell *v;       // [G + 1] the layer, updated in place; v[-1] holds -inf
  float *arate;     // [LS] the costs with an allowed option, ascending: served rate
  int *akey;        // [LS] (cost << 16) | (option index + 1)
  int *aoff;        // [LS] 16 x cost, the byte offset of V[g - cost] below V[g]
  int16_t *choice;  // [K][G + 1] option index, -1 = empty, -2 = none
};

// Listed-cost arrays: G costs at most and 8 entries of padding, rounded up to
// a multiple of 4 (16-byte reads).
__device__ __host__ inline int lex_cost_stride(int G) { return (G + 8 + 3) & ~3; }

// Options of a class are numbered by TP index, then replicas:
// q = optoff[t] + r - 1.  TP index, degree and replicas of option q.
__device__ __forceinline__ void option_of(const DevProblem &P, int q, int *ti, int *t, int *r) {
  int i = 0, first = 0, deg = P.tp[0];
  for (int t2 = 1; t2 < P.NT; ++t2) {
    if (q >= P.optoff[t2]) {  // uniform loads, per-lane selects
      i = t2;
      first = P.optoff[t2];
      deg = P.tp[t2];
    }
  }
  *ti = i;
  *t = deg;
  *r = q - first + 1;
}

// One layer suffices: V_k[g] reads V_{k+1} at budgets <= g only, so the
// budgets are rewritten from the top down, 64 at a time (lane l takes
// g = top - l), every lane's reads of a group before its writes.
//
// The preference (larger goodput, then fewer GPUs, then the earlier option,
// the empty one first) is one comparison of the goodput and one of an
// integer key: (GPUs << 16) | (option index + 1), 0 for the empty option,
// which is the entry's key plus the listed cost's (GPUs and option indices
// stay below 2^15 and 2^16).  No allowed completion is a goodput of -inf:
// it loses to every allowed one, and a budget where nothing is allowed ends
// with -inf (written as "none").  A term whose cost exceeds the budget reads
// V[-1] (-inf) through a clamped offset, so no term needs a mask.
__device__ void wave_lex_stage(const DevProblem &P, const int8_t *__restrict__ bmap, const Realisation &R,
                               int tau, int floors_met, const LexLds &X, const WaveAlloc &alloc,
                               float *goodput, double *goodput64) {
  const int lane = threadIdx.x & (kWave - 1);
  const int K = P.K, G = P.G, NT = P.NT;
  const double NEG = -__builtin_inf();
  for (int g = lane; g <= G; g += kWave) X.v[g] = LexCell{0.0, 0, 0};
  if (lane == 0) X.v[-1] = LexCell{NEG, 0, 0};
  const char *vbase = reinterpret_cast<const char *>(X.v);
  for (int k = K - 1; k >= 0; --k) {
    const bool restricted = P.has_floor && floors_met && (P.floor_rps[k] > 0.0f);
    const bool empty_ok = !restricted && tau <= 0;
    const float slo = P.slo[k], demand = P.demand[k], fl = P.floor_rps[k];
    const double rcp = P.rcp_demand[k];
    // per cost the best allowed option (served rate, then the first in
    // (TP, replicas) order), listed for the costs that have one (a ballot per
    // 64 costs)
    int n_c = 0;
    for (int c0 = 1; c0 <= G; c0 += kWave) {
      const int c = c0 + lane;
      float best = 0.0f;
      int bq = -1;
      for (int ti = 0; ti < NT && c <= G; ++ti) {  // options of cost c in (TP, replicas) order
        const int t = P.tp[ti], r = c / t;
        if (r * t != c) continue;
        const int b = bmap[k * (G + 1) + r];
        if (b < 0) continue;
        const int cell = cell_of(P, k, ti, b);
        const float cc = R.c(cell), l = R.l(cell);
        bool ok = ratio_bits(cc, l, r, slo, rcp) >= tau;
        if (restricted && !floor_ok(cc, l, r, slo, demand, fl)) ok = false;
        if (!ok) continue;
        const float sv = (l <= slo) ? served_rps(cc, r, demand) : 0.0f;
        if (bq < 0 || sv > best) {
          best = sv;
          bq = P.optoff[ti] + r - 1;
        }
      }
      const uint64_t m = __builtin_amdgcn_ballot_w64(bq >= 0);
      if (bq >= 0) {
        const int at = n_c + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
        X.arate[at] = best;
        X.akey[at] = (c << 16) | (bq + 1);
        X.aoff[at] = 16 * c;
      }
      n_c += __builtin_popcountll(m);
    }
    if (lane < 8) {  // padding: a cost no budget reaches
      X.arate[n_c + lane] = 0.0f;
      X.akey[n_c + lane] = 0;
      X.aoff[n_c + lane] = 16 * (G + 1);
    }
    __syncthreads();
    // budgets 1..G in groups of 64 (one group when G is 64); budget 0 takes
    // no listed cost, only the empty option, and is rewritten after every
    // group has read it
    for (int top = G; top >= 1; top -= kWave) {
      const int g = top - lane;
      const int gs = g >= 1 ? g : top;  // lanes past g = 1 compute nothing (valid reads)
      const LexCell e0 = X.v[gs];
      double bgp = empty_ok ? e0.gp : NEG;
      int bkey = empty_ok ? e0.key : INT_MAX;
      // listed costs up to top: the first nuse (ascending)
      int nuse = 0;
      for (int xb = 0; xb < n_c; xb += kWave) {
        const int x = xb + lane;
        const int m = __builtin_popcountll(__builtin_amdgcn_ballot_w64(x < n_c && X.aoff[min(x, n_c)] <= 16 * top));
        nuse += m;
        if (m < kWave) break;
      }
      // eight terms at a time (the preference is a total order, so the
      // order of the terms does not matter); past nuse (up to 7 entries):
      // costs above top or the padding, both reading -inf
      const int goff = 16 * gs;
      for (int x = 0; x < nuse; x += 8) {
        float ra[8];
        int ka[8], oa[8];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const float4 r4 = *reinterpret_cast<const float4 *>(X.arate + x + 4 * h);
          const int4 k4 = *reinterpret_cast<const int4 *>(X.akey + x + 4 * h);
          const int4 o4 = *reinterpret_cast<const int4 *>(X.aoff + x + 4 * h);
          ra[4 * h] = r4.x; ra[4 * h + 1] = r4.y; ra[4 * h + 2] = r4.z; ra[4 * h + 3] = r4.w;
          ka[4 * h] = k4.x; ka[4 * h + 1] = k4.y; ka[4 * h + 2] = k4.z; ka[4 * h + 3] = k4.w;
          oa[4 * h] = o4.x; oa[4 * h + 1] = o4.y; oa[4 * h + 2] = o4.z; oa[4 * h + 3] = o4.w;
        }
        LexCell vv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) vv[u] = *reinterpret_cast<const LexCell *>(vbase + max(goff - oa[u], -16));
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const double v = (double)ra[u] + vv[u].gp;
          const int key = ka[u] + vv[u].key;
          const bool better = v > bgp || (v == bgp && key < bkey);
          bgp = better ? v : bgp;
          bkey = better ? key : bkey;
        }
      }
      wave_lds_fence();
      if (g >= 1) {
        const bool none = bgp == NEG;
        X.v[g] = LexCell{bgp, none ? 0 : (bkey & ~0xFFFF), 0};
        X.choice[k * (G + 1) + g] = (int16_t)(none ? -2 : (bkey & 0xFFFF) - 1);
      }
      wave_lds_fence();
    }
    if (lane == 0) {  // budget 0: the empty option, when allowed and completed
      const LexCell e0 = X.v[0];
      const bool none = !empty_ok || e0.gp == NEG;
      X.v[0] = none ? LexCell{NEG, 0, 0} : e0;
      X.choice[k * (G + 1)] = (int16_t)(none ? -2 : -1);
    }
    __syncthreads();
  }
  if (lane == 0) {
    int rem = G;
    float gp = 0.0f;
    for (int k = 0; k < K; ++k) {
      const int q = X.choice[k * (G + 1) + rem];
      int ti_sel = -1, r_sel = 0;
      if (q >= 0) {
        int t;
        option_of(P, q, &ti_sel, &t, &r_sel);
        rem -= t * r_sel;
        const int cell = cell_of(P, k, ti_sel, bmap[k * (G + 1) + r_sel]);
        gp += served_rps(R.c(cell), r_sel, P.demand[k]);
      }
      alloc.tp_index[k] = ti_sel;
      alloc.replicas[k] = r_sel;
    }
    *goodput = gp;
    const double top_gp = X.v[G].gp;
    *goodput64 = top_gp == NEG ? 0.0 : top_gp;  // no allowed completion: 0
  }
  __syncthreads();
}

// Work area of a lexicographic solve, shared in turn by the max-min solver
// (3 (G + 1) ints) and the stage: the layer (with v[-1]), the listed costs
// and the choices, from a 16-byte aligned start.
__device__ __host__ inline size_t lex_work_bytes(int K, int G) {
  const size_t g1 = (size_t)G + 1;
  const size_t b = 16 * (g1 + 1) + 12 * (size_t)lex_cost_stride(G) + (size_t)K * g1 * sizeof(int16_t);
  const size_t solver = 3 * g1 * sizeof(int);
  return 16 + (b > solver ? b : solver);  // 16: aligning the start
}

__device__ __forceinline__ LexLds lex_lds(const DevProblem &P, void *start) {
  const size_t g1 = (size_t)P.G + 1;
  const int LS = lex_cost_stride(P.G);
  char *base = align16(start);
  LexLds X;
  X.v = reinterpret_cast<LexCell *>(base) + 1;
  X.arate = reinterpret_cast<float *>(X.v + g1);
  X.akey = reinterpret_cast<int *>(X.arate + LS);
  X.aoff = X.akey + LS;
  X.choice = reinterpret_cast<int16_t *>(X.aoff + LS);
  return X;
}

// Dense batch under the whole objective: one wavefront per scenario.
// STAGE: inputs staged in LDS (1) or read from global memory (0), fixed at
// compile time so that every access compiles for its own memory.
template <int STAGE>
__global__ __launch_bounds__(64) void k_solve_dense_lex(DevProblem P, const int8_t *__restrict__ bmap,
                                                        const float *__restrict__ cap,
                                                        const float *__restrict__ tail, int64_t n,
                                                        AllocOut out, double *__restrict__ gp64_out) {
  constexpr int stage = STAGE;
  extern __shared__ int lds[];
  const int64_t j = blockIdx.x;
  if (j >= n) return;
  int *tp_index = lds;
  int *replicas = tp_index + kMaxClasses;
  int *work = replicas + kMaxClasses;
  WaveAlloc wa{tp_index, replicas};
  const LexLds X = lex_lds(P, work);
  Realisation R{cap + j * P.N, tail + j * P.N, -1, 0.0f, 0.0f};
  if (stage) {
    const StageArea A = stage_area(P, reinterpret_cast<char *>(work) + lex_work_bytes(P.K, P.G));
    stage_copy_bmap(P, bmap, A.bmap);
    stage_copy_cells(P, R.cap, R.tail, A.cap, A.tail);
    bmap = A.bmap;
    R.cap = A.cap;
    R.tail = A.tail;
    __syncthreads();
  }
  int fm;
  float gp;
  double gp64;
  const int tau = wave_solve(P, bmap, R, work, &fm, nullptr, nullptr);
  wave_lex_stage(P, bmap, R, tau, fm, X, wa, &gp, &gp64);
  write_alloc(out, j, P.K, tau, fm, gp, wa);
  if (gp64_out && threadIdx.x == 0) gp64_out[j] = gp64;
}

// Certificate with the stage-wise gap: both allocations under the whole
// objective; max-min gap tau+ - tau-, goodput gap |gp+ - gp-| / max(gp+,
// gp-) (0 when both are 0); within eps means both stages are.  Block (R, o)
// solves realisation R of order o (0: conservative, 1: optimistic) and
// keeps its result in a record; k_certify_state then takes each
// order's gaps and state from the two records.
// STAGE: inputs staged in LDS (1) or read from global memory (0), fixed at
// compile time so that every access compiles for its own memory.
template <int STAGE>
__global__ __launch_bounds__(64) void k_certify_lex(DevProblem P, const int8_t *__restrict__ bmap,
                                                    const float *__restrict__ cap_lo,
                                                    const float *__restrict__ cap_hi,
                                                    const float *__restrict__ tail_lo,
                                                    const float *__restrict__ tail_hi, AllocOut cons,
                                                    AllocOut opt, CertRec *__restrict__ rec) {
  constexpr int stage = STAGE;
  extern __shared__ int lds[];
  const int R = blockIdx.x, o = blockIdx.y;
  const size_t off = (size_t)o * P.N;
  int *t_index = lds;
  int *t_rep = t_index + kMaxClasses;
  int *work = t_rep + kMaxClasses;
  WaveAlloc wa{t_index, t_rep};
  const LexLds X = lex_lds(P, work);
  const StageArea A = stage_area(P, reinterpret_cast<char *>(work) + lex_work_bytes(P.K, P.G));
  const int8_t *bm = bmap;
  Realisation rz = R == 0 ? Realisation{cap_lo + off, tail_hi + off, -1, 0.0f, 0.0f}
                          : Realisation{cap_hi + off, tail_lo + off, -1, 0.0f, 0.0f};
  if (stage) {
    stage_copy_bmap(P, bmap, A.bmap);
    stage_copy_cells(P, rz.cap, rz.tail, A.cap, A.tail);
    bm = A.bmap;
    rz = Realisation{A.cap, A.tail, -1, 0.0f, 0.0f};
    __syncthreads();
  }
  int fm;
  float gp;
  double g64;
  const int tau = wave_solve(P, bm, rz, work, &fm, nullptr, nullptr);
  wave_lex_stage(P, bm, rz, tau, fm, X, wa, &gp, &g64);
  write_alloc(R == 0 ? cons : opt, o, P.K, tau, fm, gp, wa);
  write_cert_rec(rec + (size_t)o * 2 + R, P.K, tau, fm, gp, g64, wa);
}


// ---------------------------------------------------------------------------
// The acquisition score with the stage-wise gap under the whole objective:
// per scenario both allocations by the max-min solver and level (3)'s
// knapsack, Gamma_mm = tau+ - tau- and Gamma_gp = |gp+ - gp-| / max(gp+,
// gp-); the expected reduction of each stage per (order, candidate); the
// argmax by the max-min stage, then the goodput stage, then the cost order.
// Block (chunk, e, o) takes samples [64 chunk, 64 chunk + 64) one after
// another with the whole wavefront; lane j keeps sample j's two gaps.
// ---------------------------------------------------------------------------
__device__ __host__ inline size_t stage2_bytes(const DevProblem &P) {  // bucket map + two realisations
  return 16 + (((size_t)P.K * (P.G + 1) + 3) & ~(size_t)3) + 4 * sizeof(float) * (size_t)P.N;
}

__device__ __forceinline__ void stage_gaps(int tau_m, int tau_p, double gm, double gp, double *mm, double *gg) {
  *mm = (double)__int_as_float(tau_p) - (double)__int_as_float(tau_m);
  const double top = gp > gm ? gp : gm;
  *gg = top > 0.0 ? fabs(gp - gm) / top : 0.0;
}

// STAGE: inputs staged in LDS (1) or read from global memory (0), fixed at
// compile time so that every access compiles for its own memory.
template <int STAGE>
__global__ __launch_bounds__(64) void k_score_lex_wave(DevProblem P, const int8_t *__restrict__ bmap,
                                                       const CandInfo *__restrict__ info,
                                                       const float *__restrict__ cap_lo,
                                                       const float *__restrict__ cap_hi,
                                                       const float *__restrict__ tail_lo,
                                                       const float *__restrict__ tail_hi,
                                                       const uint8_t *__restrict__ measured,
                                                       const float *__restrict__ cap_s,
                                                       const float *__restrict__ tail_s, int32_t E, int32_t S,
                                                       double *__restrict__ part_mm, double *__restrict__ part_gp,
                                                       int64_t n_partial) {
  constexpr int stage = STAGE;
  extern __shared__ int lds[];
  const int chunk = blockIdx.x, e = blockIdx.y, o = blockIdx.z;
  const int lane = threadIdx.x;
  const CandInfo ci = info[e];
  const size_t tile = (size_t)o * E + e;
  const size_t off = (size_t)o * P.N;
  if (ci.cls < 0 || measured[off + ci.cell]) return;  // not scored (the finalize writes those)
  int *tpi = lds;
  int *rep = tpi + kMaxClasses;
  int *work = rep + kMaxClasses;
  WaveAlloc wa{tpi, rep};
  const LexLds X = lex_lds(P, work);
  const int8_t *bm = bmap;
  const float *cm = cap_lo + off, *lm = tail_hi + off, *cp = cap_hi + off, *lp = tail_lo + off;
  if (stage) {
    char *st = reinterpret_cast<char *>(work) + lex_work_bytes(P.K, P.G);
    int8_t *sb = reinterpret_cast<int8_t *>(align16(st));
    float *sc = reinterpret_cast<float *>(sb + (((size_t)P.K * (P.G + 1) + 3) & ~(size_t)3));
    stage_copy_bmap(P, bmap, sb);
    stage_copy_cells(P, cm, lm, sc, sc + P.N);
    stage_copy_cells(P, cp, lp, sc + 2 * P.N, sc + 3 * P.N);
    bm = sb;
    cm = sc;
    lm = sc + P.N;
    cp = sc + 2 * P.N;
    lp = sc + 3 * P.N;
    __syncthreads();
  }
  double mine_mm = 0.0, mine_gp = 0.0;
  const int s0 = chunk * kWave;
  const int ns = min(kWave, S - s0);
  for (int j = 0; j < ns; ++j) {
    const float cs = cap_s[tile * S + s0 + j];
    const float ts = tail_s[tile * S + s0 + j];
    int fm;
    float g32;
    double gm, gp;
    Realisation rm{cm, lm, ci.cell, cs, ts};
    const int tm = wave_solve(P, bm, rm, work, &fm, nullptr, nullptr);
    wave_lex_stage(P, bm, rm, tm, fm, X, wa, &g32, &gm);
    Realisation rp{cp, lp, ci.cell, cs, ts};
    const int tp = wave_solve(P, bm, rp, work, &fm, nullptr, nullptr);
    wave_lex_stage(P, bm, rp, tp, fm, X, wa, &g32, &gp);
    // the binary64 totals are in lane 0
    gm = __hiloint2double(__builtin_amdgcn_readfirstlane(__double2hiint(gm)),
                          __builtin_amdgcn_readfirstlane(__double2loint(gm)));
    gp = __hiloint2double(__builtin_amdgcn_readfirstlane(__double2hiint(gp)),
                          __builtin_amdgcn_readfirstlane(__double2loint(gp)));
    double mm, gg;
    stage_gaps(tm, tp, gm, gp, &mm, &gg);
    if (lane == j) {
      mine_mm = mm;
      mine_gp = gg;
    }
  }
  const double sum_mm = wave_pairwise_sum(mine_mm);
  const double sum_gp = wave_pairwise_sum(mine_gp);
  if (lane == 0) {
    part_mm[tile * n_partial + chunk] = sum_mm;
    part_gp[tile * n_partial + chunk] = sum_gp;
  }
}

// ---------------------------------------------------------------------------
// The stage-wise score's goodput stage without full solves (no critical
// floors).  Level (3) of the objective on a scenario keeps every class's
// ratio at least the scenario's tau* and maximises the total served
// goodput.  Splitting off the candidate's class i,
//   gp = max over allowed options q of class i of served_q + V_i(tau*)[G - cost_q],
// where V_i(tau)[g] is the best goodput of the other classes with at most g
// GPUs when only options of ratio >= tau are allowed (the empty option only
// when tau <= 0).  Only the candidate cell's options depend on the sample;
// V_i and the allowed set of every other option change only where tau
// crosses an option's ratio.  Over the sorted distinct ratios b_0 = 0 <
// b_1 < ... < b_{n-1} of the realisation's options (every class, every
// cell), tau* falls in interval j = #{b_m < tau*}; there the options of
// ratio >= b_j are allowed (none for j = n) and the empty option only in
// interval 0 (tau* = 0).  Per (realisation, order, class i) and interval
// the set-up tabulates V_i and, for class i's options off the candidate
// cell, the best value per cell reduced to the largest (at its cell), the
// largest over every other cell and the empty option's; a scenario then
// needs its interval (a bisection over the ratios) and its cell's options.
// Goodput sums are binary64, exact under the same condition as the full
// solve's (nonzero served rates within a factor 2^23 of each other), so the
// association does not change them.
// ---------------------------------------------------------------------------
constexpr int kLexPrepThreads = 256;
// Wavefronts of the interval tables kernel in all (blocks per realisation,
// order and class follow from it, no more than the intervals can use): a
// wavefront walks its intervals one after another, so more and shorter-lived
// wavefronts shorten the kernel, until they take the SIMDs from the
// certificate solves running beside it on the second stream (on 4 classes at
// G = 64 the whole call took 86.1-86.2, 81.8-83.8 and 83.4 us with 8192,
// 12288 and 16384).
constexpr int kLexTableWaves = 12288;

// Keys the breakpoint sort takes: every option's ratio and the 0, padded to
// a power of two (at least one per thread).
__host__ __device__ inline int lex_sort_keys(int nopt) {
  int n = kLexPrepThreads;
  while (n < nopt + 1) n <<= 1;
  return n;
}

// LDS of a breakpoint block: the sort keys, one count per thread and the
// realisation's cells (capacity and tail).
__host__ __device__ inline size_t lex_breaks_lds(int nopt, int N) {
  return 4 * ((size_t)lex_sort_keys(nopt) + kLexPrepThreads) + 8 * (size_t)N;
}

// LDS of a k_lex_tables block: every option's (ratio, served rate), the
// candidate class's options (cost, cell), then (from a 16-byte boundary)
// per wavefront two knapsack layers (binary64, each with G + 1 entries of
// padding), one class's best served rates (binary64) and its listed costs,
// G + 8 of each rounded up to a multiple of 4.
__host__ __device__ inline int lex_list_stride(int G) { return (G + 8 + 3) & ~3; }
__host__ __device__ inline size_t lex_tables_head(int nopt, int per_class_options) {
  return (8 * ((size_t)nopt + per_class_options) + 15) & ~(size_t)15;
}
__host__ __device__ inline size_t lex_tables_lds(int nopt, int per_class_options, int G) {
  const size_t nw = kLexPrepThreads / kWave;
  return lex_tables_head(nopt, per_class_options) +
         nw * (16 * (2 * (size_t)G + 2) + 12 * (size_t)lex_list_stride(G));
}

// LDS of a k_score_lex_excl block: both realisations' breakpoints and M of
// the candidate's replica range.
__host__ __device__ inline size_t lex_score_lds(int nbmax, int rmax) {
  return sizeof(int) * (2 * (size_t)nbmax + 2 * (size_t)rmax);
}

// Bitonic sort of n2 = M x kLexPrepThreads keys (M = 1 or 2) held in
// registers: thread t holds positions M t .. M t + M - 1.  A stage pairs
// position p with p ^ stride; the lower one keeps the minimum when the run
// of length size it lies in ascends ((p & size) == 0), else the maximum.
// Within a wavefront (stride / M < 64) the partner's key comes by a lane
// shuffle, one round trip per stage with no LDS write or barrier (DPP row
// moves for the short distances measured slower); the stages across
// wavefronts go through keys (LDS) between block barriers.
// On return keys holds the sorted keys (block-synchronised).
template <int M>
__device__ __forceinline__ void bitonic_regs(int *keys, int n2, int tid) {
  int v[M];
#pragma unroll
  for (int j = 0; j < M; ++j) v[j] = keys[M * tid + j];
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride < M) {  // M = 2, stride 1: both positions in this thread
        const bool up = ((M * tid) & size) == 0;
        const int a = v[0], b = v[M - 1];
        v[0] = up ? min(a, b) : max(a, b);
        v[M - 1] = up ? max(a, b) : min(a, b);
      } else if (stride / M < kWave) {
#pragma unroll
        for (int j = 0; j < M; ++j) {
          const int p = M * tid + j;
          const int w = __shfl_xor(v[j], stride / M, kWave);
          const bool keep_min = ((p & stride) == 0) == ((p & size) == 0);
          v[j] = keep_min ? min(v[j], w) : max(v[j], w);
        }
      } else {
        __syncthreads();  // earlier reads of keys are done
#pragma unroll
        for (int j = 0; j < M; ++j) keys[M * tid + j] = v[j];
        __syncthreads();
#pragma unroll
        for (int j = 0; j < M; ++j) {
          const int p = M * tid + j;
          const int w = keys[p ^ stride];
          const bool keep_min = ((p & stride) == 0) == ((p & size) == 0);
          v[j] = keep_min ? min(v[j], w) : max(v[j], w);
        }
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < M; ++j) keys[M * tid + j] = v[j];
  __syncthreads();
}

// Per (realisation R, order o), one block of kLexPrepThreads threads: every
// option of every class (ratio bits, -1 when no load level holds it; served
// rate) to opt_out, and the sorted distinct ratios, 0 always among them, to
// bp_out (nb of them to nbp).  The ratios are sorted by a bitonic network in
// LDS, then each first occurrence is placed by a block-wide count of the
// ones before it.  Load levels come from the problem (the bucket map's
// values), so the block does not wait for the map.
__device__ void lex_breaks_block(const DevProblem &P, int R, int o, const float *__restrict__ cap_lo,
                                 const float *__restrict__ cap_hi, const float *__restrict__ tail_lo,
                                 const float *__restrict__ tail_hi, int32_t nbmax, int2 *__restrict__ opt_out,
                                 float *__restrict__ bp_out, int32_t *__restrict__ nbp) {
  extern __shared__ int lex_keys[];
  const int tid = threadIdx.x;
  const int K = P.K, N = P.N, B = P.B, NT = P.NT, per_class = NT * B, PP = P.optoff[NT];
  const int nopt = K * PP, n2 = lex_sort_keys(nopt);
  int *cnt = lex_keys + n2;
  float *ccap = reinterpret_cast<float *>(cnt + kLexPrepThreads), *ctail = ccap + N;
  const size_t off = (size_t)o * N;
  const float *gcap = (R == 0 ? cap_lo : cap_hi) + off;
  const float *gtail = (R == 0 ? tail_hi : tail_lo) + off;
  int2 *opt = opt_out + ((size_t)o * 2 + R) * nopt;
  // problem constants indexed per lane below, and the realisation's cells,
  // staged in one round trip (kernel arguments indexed per lane are a
  // memory load per access); the option offsets in registers
  __shared__ float s_slo[kMaxClasses], s_dm[kMaxClasses];
  __shared__ double s_rcp[kMaxClasses];
  if (tid < K) {
    s_slo[tid] = P.slo[tid];
    s_dm[tid] = P.demand[tid];
    s_rcp[tid] = P.rcp_demand[tid];
  }
  for (int c = tid; c < N; c += kLexPrepThreads) {
    ccap[c] = gcap[c];
    ctail[c] = gtail[c];
  }
  int ofr[kMaxTp];
#pragma unroll
  for (int j = 0; j < kMaxTp; ++j) ofr[j] = j < NT ? P.optoff[j] : INT_MAX;
  __syncthreads();
  for (int q = tid; q < n2; q += kLexPrepThreads) {
    int key = INT_MAX;  // padding and options that do not exist sort last
    if (q < nopt) {
      const int k = q / PP, p = q - k * PP;
      int ti = 0, first = 0;
#pragma unroll
      for (int j = 1; j < kMaxTp; ++j) {
        const bool in = p >= ofr[j];
        ti = in ? j : ti;
        first = in ? ofr[j] : first;
      }
      const int r = p - first + 1;
      const int b = level_from(P, s_dm[k] / (float)r);  // level_of with the staged demand
      const int cell = k * per_class + ti * B + max(b, 0);
      const float c = ccap[cell], l = ctail[cell];
      const int f = b >= 0 ? ratio_bits(c, l, r, s_slo[k], s_rcp[k]) : -1;
      const float sv = b >= 0 && l <= s_slo[k] ? served_rps(c, r, s_dm[k]) : 0.0f;
      if (b >= 0) key = f;
      opt[q] = make_int2(f, __float_as_int(sv));
    } else if (q == nopt) {
      key = 0;  // tau* = 0 is its own interval (the empty option's)
    }
    lex_keys[q] = key;
  }
  __syncthreads();
  if (n2 == kLexPrepThreads) {
    bitonic_regs<1>(lex_keys, n2, tid);
  } else if (n2 == 2 * kLexPrepThreads) {
    bitonic_regs<2>(lex_keys, n2, tid);
  } else {
    // Bitonic sort in LDS.  A stage of stride at most 64 pairs keys inside
    // aligned runs of 128, and one wavefront handles every pair of a run (the
    // 64 pair indices of a wavefront map to one run), so such a stage only
    // waits for its own wavefront's writes, unless the stage before it
    // crossed runs.
    int prev = n2;
    for (int size = 2; size <= n2; size <<= 1) {
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        if (stride > kWave || prev > kWave) __syncthreads();
        else wave_lds_fence();
        prev = stride;
        for (int idx = tid; idx < (n2 >> 1); idx += kLexPrepThreads) {
          const int lo = ((idx & ~(stride - 1)) << 1) | (idx & (stride - 1)), hi = lo + stride;
          const int a = lex_keys[lo], c = lex_keys[hi];
          const bool up = (lo & size) == 0;
          if ((a > c) == up) {
            lex_keys[lo] = c;
            lex_keys[hi] = a;
          }
        }
      }
    }
    __syncthreads();
  }
  // thread t owns keys [t seg, (t + 1) seg): count its first occurrences,
  // then an exclusive count over the threads places them
  const int seg = n2 / kLexPrepThreads, a0 = tid * seg;
  int mine = 0;
  for (int a = a0; a < a0 + seg; ++a) {
    const int v = lex_keys[a];
    mine += (v != INT_MAX && (a == 0 || lex_keys[a - 1] != v)) ? 1 : 0;
  }
  // inclusive scan within the wavefront, then the totals of the ones before
  const int lane = tid & (kWave - 1), wave = tid >> 6;
  int incl = mine;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int v = __shfl_up(incl, d, kWave);
    if (lane >= d) incl += v;
  }
  if (lane == kWave - 1) cnt[wave] = incl;
  __syncthreads();
  int before = incl - mine, total = 0;
  for (int w = 0; w < kLexPrepThreads / kWave; ++w) {
    before += w < wave ? cnt[w] : 0;
    total += cnt[w];
  }
  float *bp = bp_out + ((size_t)o * 2 + R) * nbmax;
  for (int a = a0; a < a0 + seg; ++a) {
    const int v = lex_keys[a];
    if (v != INT_MAX && (a == 0 || lex_keys[a - 1] != v)) bp[before++] = __int_as_float(v);
  }
  if (tid == 0) nbp[o * 2 + R] = total;
}

// A call's set-up in one launch of kLexPrepThreads-thread blocks: blocks
// [0, nb) the bucket map (one entry per thread), [nb, nb + nc) the candidate
// records (one per thread), then n_br blocks of option ratios and
// breakpoints, block 2 o + R for realisation R of order o.  The parts are
// independent: each takes the load levels from the problem.
__global__ __launch_bounds__(kLexPrepThreads) void k_setup(DevProblem P, int8_t *__restrict__ bmap, int32_t nb,
                                                          const int32_t *__restrict__ cand, int32_t E,
                                                          CandInfo *__restrict__ info, int32_t nc,
                                                          const float *__restrict__ cap_lo,
                                                          const float *__restrict__ cap_hi,
                                                          const float *__restrict__ tail_lo,
                                                          const float *__restrict__ tail_hi, int32_t nbmax,
                                                          int2 *__restrict__ opt_out, float *__restrict__ bp_out,
                                                          int32_t *__restrict__ nbp) {
  const int b = blockIdx.x;
  if (b < nb) {
    setup_bucket_at(P, bmap, b * kLexPrepThreads + (int)threadIdx.x);
    return;
  }
  if (b < nb + nc) {
    setup_cand_at(P, cand, E, info, (b - nb) * kLexPrepThreads + (int)threadIdx.x);
    return;
  }
  const int z = b - nb - nc;
  lex_breaks_block(P, z & 1, z >> 1, cap_lo, cap_hi, tail_lo, tail_hi, nbmax, opt_out, bp_out, nbp);
}

// Per (realisation R, order o, class i) and interval j of the breakpoints
// (one wavefront each): V_i, the best goodput of the classes other than i
// with at most g GPUs, g = 0..G, when only options of ratio >= bp[j] are
// allowed (none when j = nb) and the empty option only when j = 0; then
// class i's best served + V_i[G - cost] per cell, reduced to the largest
// (and its cell), the largest over the other cells, and the empty
// option's.  The knapsack takes the classes from the last to the first
// with a best-served-per-cost vector each (the options of one cost merged):
//   V'[g] = max(V[g] if empty allowed, max_{c=1..g} A[c] + V[g - c]),
// lanes over g from the top down, so each chunk loops c only up to its
// largest g.  Blocks split the intervals of one (R, o, i) four wavefronts
// at a time.
template <int NTP>
__global__ __launch_bounds__(kLexPrepThreads) void k_lex_tables(DevProblem P, const int8_t *__restrict__ bmap,
                                                               const int2 *__restrict__ opt_in,
                                                               const float *__restrict__ bp_in,
                                                               const int32_t *__restrict__ nbp, int32_t nbmax,
                                                               int32_t nsplit, double *__restrict__ Vout,
                                                               double *__restrict__ Wout) {
  extern __shared__ __attribute__((aligned(16))) double lex_tab_lds[];  // 16-byte reads below
  const int R = blockIdx.x & 1, part = blockIdx.x >> 1, o = blockIdx.y, i = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  constexpr int nw = kLexPrepThreads / kWave;
  const int K = P.K, G = P.G, B = P.B, NT = P.NT, PP = P.optoff[NT];
  const int nopt = K * PP;
  const int nb = nbp[o * 2 + R];
  const int first = part * nw + wave, step = nsplit * nw;
  int2 *oinfo = reinterpret_cast<int2 *>(lex_tab_lds);  // [nopt] ratio bits, served rate bits
  int2 *icost = oinfo + nopt;                            // [PP] class i's options: cost, cell
  // per wavefront two knapsack layers, each with G + 1 entries of -inf
  // below index 0, so that V[g - c] for a cost above the budget reads -inf
  // (which the max ignores) instead of needing a clamp and a mask
  double *vreg = reinterpret_cast<double *>(reinterpret_cast<char *>(lex_tab_lds) + lex_tables_head(nopt, PP));
  double *Va = vreg + (size_t)wave * 2 * (2 * G + 2) + (G + 1);
  double *Vb = Va + 2 * G + 2;
  // per wavefront: the costs with an allowed option (as byte offsets into a
  // layer) and their best served rates, ascending, then padding
  const int LS = lex_list_stride(G);
  double *Ad = vreg + (size_t)nw * 2 * (2 * G + 2) + (size_t)wave * LS;
  int *Ck = reinterpret_cast<int *>(vreg + (size_t)nw * 2 * (2 * G + 2) + (size_t)nw * LS) + (size_t)wave * LS;
  if (part * nw > nb) return;  // no interval for this block
  const int2 *opt = opt_in + ((size_t)o * 2 + R) * nopt;
  for (int q = tid; q < nopt; q += kLexPrepThreads) oinfo[q] = opt[q];
  // class i's options: (cost, cell within the class; -1 when no level holds
  // it); TP decode from staged constants
  __shared__ int s_tp[kMaxTp], s_off[kMaxTp + 1];
  if (tid < NT) s_tp[tid] = P.tp[tid];
  if (tid <= NT) s_off[tid] = P.optoff[tid];
  __syncthreads();
  for (int p = tid; p < PP; p += kLexPrepThreads) {
    int ti = 0;
    while (ti + 1 < NT && p >= s_off[ti + 1]) ++ti;
    const int r = p - s_off[ti] + 1;
    const int b = bmap[i * (G + 1) + r];
    icost[p] = make_int2(s_tp[ti] * r, b >= 0 ? ti * B + b : -1);
  }
  __syncthreads();
  const double NEG = -__builtin_inf();
  const float NEGF = -__builtin_inff();
  // the TP degrees, their reciprocals and option offsets in registers
  int tpr[NTP], ofr[NTP];
  float tpinv[NTP];
#pragma unroll
  for (int ti = 0; ti < NTP; ++ti) {
    tpr[ti] = ti < NT ? P.tp[ti] : 0;
    ofr[ti] = ti < NT ? P.optoff[ti] : 0;
    tpinv[ti] = tpr[ti] > 0 ? 1.0f / (float)tpr[ti] : 0.0f;
  }
  for (int g = lane; g <= G; g += kWave) {  // the padding below index 0, never written again
    Va[-1 - g] = NEG;
    Vb[-1 - g] = NEG;
  }
  const float *bp = bp_in + ((size_t)o * 2 + R) * nbmax;
  const size_t row0 = (((size_t)o * 2 + R) * K + i) * (size_t)(nbmax + 1);
  for (int j = first; j <= nb; j += step) {
    const int thr = j < nb ? __float_as_int(bp[j]) : INT_MAX;  // allowed: ratio >= thr
    const bool empty_ok = j == 0;
    for (int g = lane; g <= G; g += kWave) Va[g] = 0.0;  // no class yet: nothing served
    wave_lds_fence();
    double *Vp = Va, *Vc = Vb;
    for (int k = K - 1; k >= 0; --k) {
      if (k == i) continue;
      // A[c]: the best served rate of class k's allowed options of cost c,
      // listed only for the costs that have one (a ballot per 64 costs).
      // The options of cost c are (t, c / t) for the TP degrees t dividing
      // c; every degree's read is issued (at option 0 when t does not
      // divide c), so they overlap.
      int n_c = 0;
      for (int c0 = 1; c0 <= G; c0 += kWave) {
        const int c = c0 + lane;
        int2 ov[NTP];
        bool okv[NTP];
#pragma unroll
        for (int ti = 0; ti < NTP; ++ti) {
          // c / t, exact whenever t divides c (the float quotient is within
          // 1/2 of it for c <= 2^22)
          const int r = (int)((float)c * tpinv[ti] + 0.5f);
          okv[ti] = (ti < NT) & (c <= G) & (r >= 1) & (r * tpr[ti] == c);  // no short-circuit branches
          ov[ti] = oinfo[okv[ti] ? k * PP + ofr[ti] + r - 1 : 0];
        }
        float a = NEGF;
#pragma unroll
        for (int ti = 0; ti < NTP; ++ti)
          a = okv[ti] && ov[ti].x >= thr ? fmaxf(a, __int_as_float(ov[ti].y)) : a;
        const bool has = a > NEGF;
        const uint64_t m = __builtin_amdgcn_ballot_w64(has);
        if (has) {
          const int at = n_c + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
          Ad[at] = (double)a;
          Ck[at] = 8 * c;
        }
        n_c += __builtin_popcountll(m);
      }
      if (lane < 8) {  // padding: a cost no budget reaches
        Ck[n_c + lane] = 8 * (G + 1);
        Ad[n_c + lane] = 0.0;
      }
      wave_lds_fence();
      // V'[g] = max(V[g] if empty allowed, max over listed c <= g of A[c] + V[g - c]):
      // the max is exact, so the order of the terms does not matter, and a
      // term with c > g reads the padding (-inf; A[c] + -inf is -inf), so
      // any superset of the terms c <= g gives the same value.  A lane reads
      // V[g - c] at its own V[g] minus c's byte offset, and the costs and
      // rates eight at a time (16-byte reads at the same address in every
      // lane): per term one subtraction, one addition and one maximum, and
      // per eight terms two round trips to LDS.
      // budget 0 takes no listed cost (costs are at least 1); budgets 1..G
      // in groups of 64 (one group when G is 64)
      if (lane == 0) Vc[0] = empty_ok ? Vp[0] : NEG;
      for (int top = G; top >= 1; top -= kWave) {
        const int g = top - lane;  // lanes past g = 1 compute nothing
        const int gs = g >= 0 ? g : 0;
        const char *vg = reinterpret_cast<const char *>(Vp + gs);
        double best = empty_ok ? Vp[gs] : NEG;
        // listed costs up to top: the first nuse (ascending)
        int nuse = 0;
        for (int xb = 0; xb < n_c; xb += kWave) {
          const int x = xb + lane;
          const int m = __builtin_popcountll(__builtin_amdgcn_ballot_w64(x < n_c && Ck[min(x, n_c)] <= 8 * top));
          nuse += m;
          if (m < kWave) break;
        }
        // past nuse (up to 7 entries): listed costs above top or the padding
        // (cost G + 1, at most G + 1 below index 0), both reading -inf here
        for (int x = 0; x < nuse; x += 8) {
          int cq[8];
          double aq[8], vq[8];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int4 c4 = *reinterpret_cast<const int4 *>(Ck + x + 4 * h);
            const double2 a01 = *reinterpret_cast<const double2 *>(Ad + x + 4 * h);
            const double2 a23 = *reinterpret_cast<const double2 *>(Ad + x + 4 * h + 2);
            cq[4 * h] = c4.x; cq[4 * h + 1] = c4.y; cq[4 * h + 2] = c4.z; cq[4 * h + 3] = c4.w;
            aq[4 * h] = a01.x; aq[4 * h + 1] = a01.y; aq[4 * h + 2] = a23.x; aq[4 * h + 3] = a23.y;
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) vq[u] = *reinterpret_cast<const double *>(vg - cq[u]);
#pragma unroll
          for (int u = 0; u < 8; ++u) best = fmax(best, aq[u] + vq[u]);
        }
        if (g >= 1) Vc[g] = best;
      }
      wave_lds_fence();
      double *t2 = Vp;
      Vp = Vc;
      Vc = t2;
    }
    double *Vg = Vout + (row0 + j) * (size_t)(G + 1);
    for (int g = lane; g <= G; g += kWave) Vg[g] = Vp[g];
    // class i's allowed options: served + V[G - cost], reduced to the
    // largest value w1 (with a cell c1 holding it) and w2, the largest over
    // the cells other than c1.  Merging two such summaries: same c1, the
    // larger of each; else the larger w1 leads and the other's w1 (from
    // another cell) competes for w2.  Lanes over the options, then a
    // butterfly (the merge is symmetric, so every lane ends with the same).
    double w1 = NEG, w2 = NEG;
    int c1 = -1;
    auto merge = [&](double b1, int bc, double b2) {
      if (bc == c1) {
        w1 = fmax(w1, b1);
        w2 = fmax(w2, b2);
      } else if (b1 > w1 || (b1 == w1 && bc > c1)) {
        w2 = fmax(b2, w1);
        w1 = b1;
        c1 = bc;
      } else {
        w2 = fmax(w2, b1);
      }
    };
    for (int p = lane; p < PP; p += kWave) {
      const int2 ic = icost[p];
      const int2 ov = oinfo[i * PP + p];
      if (ic.y >= 0 && ov.x >= thr) merge((double)__int_as_float(ov.y) + Vp[G - ic.x], ic.y, NEG);
    }
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) {
      const double o1 = __shfl_xor(w1, m, kWave), o2 = __shfl_xor(w2, m, kWave);
      const int oc = __shfl_xor(c1, m, kWave);
      merge(o1, oc, o2);
    }
    if (lane == 0) {
      double *Wj = Wout + (row0 + j) * 4;
      Wj[0] = w1;
      Wj[1] = w2;
      Wj[2] = empty_ok ? Vp[G] : NEG;
      Wj[3] = (double)c1;
    }
    wave_lds_fence();
  }
}

// Scenarios of the stage-wise score without full solves: block (chunk of 64
// samples, candidate, order), lane = sample.  Per realisation tau* by the
// exclusion identity of the max-min score (U, and M of the range's options),
// its interval among the breakpoints (bisection in LDS), then
// gp = max(the class's best off the candidate cell, the empty option, the
// candidate cell's allowed options at the sample: served + V[G - cost]);
// both stages' gaps reduced by the pairwise wave tree, one partial each.
__global__ __launch_bounds__(64) void k_score_lex_excl(DevProblem P, const TileInfo *__restrict__ tiles,
                                                       const int32_t *__restrict__ mopt, int32_t n_thr,
                                                       const float *__restrict__ cap_s,
                                                       const float *__restrict__ tail_s, int32_t E, int32_t S,
                                                       const float *__restrict__ bp, const int32_t *__restrict__ nbp,
                                                       int32_t nbmax, int32_t rmax, const double *__restrict__ V,
                                                       const double *__restrict__ W, double *__restrict__ part_mm,
                                                       double *__restrict__ part_gp, int64_t n_partial) {
  extern __shared__ int lex_bp[];  // [2][nbmax] breakpoints, then [2][rmax] M of the range
  int *Ml = lex_bp + 2 * nbmax;
  const int chunk = blockIdx.x, e = blockIdx.y, o = blockIdx.z, lane = threadIdx.x;
  const size_t tile = (size_t)o * E + e;
  // the loads that need nothing else come first, together: the tile
  // record, both realisations' breakpoints (every slot; those past the
  // count are not used), the lane's sample
  const TileInfo tl = tiles[tile];
  const int nb0 = nbp[o * 2 + 0], nb1 = nbp[o * 2 + 1];
  for (int m = lane; m < nbmax; m += kWave) {
    lex_bp[m] = __float_as_int(bp[((size_t)o * 2 + 0) * nbmax + m]);
    lex_bp[nbmax + m] = __float_as_int(bp[((size_t)o * 2 + 1) * nbmax + m]);
  }
  const int s = chunk * kWave + lane;
  const bool live = s < S;
  const float cs = cap_s[tile * S + (live ? s : 0)];
  const float ls = tail_s[tile * S + (live ? s : 0)];
  if (tl.state != 0) return;  // measured or invalid: the finalize writes those
  // M of the range's options, both realisations, into LDS
  const int nr = tl.rhi >= tl.rlo ? tl.rhi - tl.rlo + 1 : 0;
  for (int j = lane; j < nr; j += kWave) {
    Ml[j] = mopt[((size_t)o * 2 + 0) * n_thr + tl.toff + j];
    Ml[rmax + j] = mopt[((size_t)o * 2 + 1) * n_thr + tl.toff + j];
  }
  wave_lds_fence();
  const int G = P.G, K = P.K, per_class = P.NT * P.B;
  const int i = tl.cls, local = tl.cell - i * per_class;
  const float slo = P.slo[i], lam = P.demand[i];
  const double rcp = P.rcp_demand[i];
  // tau* and its interval, both realisations
  int tau[2], row_j[2];
#pragma unroll
  for (int R = 0; R < 2; ++R) {
    int t = R == 0 ? tl.u_m : tl.u_p;
    for (int r = tl.rlo; r <= tl.rhi; ++r) t = max(t, min(ratio_bits(cs, ls, r, slo, rcp), Ml[R * rmax + r - tl.rlo]));
    tau[R] = t;
    // interval: the count of breakpoints below tau
    const int nb = R == 0 ? nb0 : nb1;
    const int *b = lex_bp + R * nbmax;
    int lo = 0, hi = nb;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (b[mid] < t) lo = mid + 1;
      else hi = mid;
    }
    row_j[R] = lo;
  }
  // the interval tables of both realisations: the summary first (both
  // rows' loads together), then the candidate cell's allowed options
  const double *Wj[2], *Vj[2];
  double w[2][4];
#pragma unroll
  for (int R = 0; R < 2; ++R) {
    const size_t row = ((((size_t)o * 2 + R) * K + i) * (size_t)(nbmax + 1) + row_j[R]);
    Wj[R] = W + row * 4;
    Vj[R] = V + row * (size_t)(G + 1);
#pragma unroll
    for (int q = 0; q < 4; ++q) w[R][q] = Wj[R][q];
  }
  double gp[2];
#pragma unroll
  for (int R = 0; R < 2; ++R) {
    double g = (int)w[R][3] == local ? w[R][1] : w[R][0];
    gp[R] = fmax(g, w[R][2]);
  }
  for (int r = tl.rlo; r <= tl.rhi; ++r) {
    const int f = ratio_bits(cs, ls, r, slo, rcp);
    const float sv = ls <= slo ? served_rps(cs, r, lam) : 0.0f;
    const double v0 = Vj[0][G - tl.t * r], v1 = Vj[1][G - tl.t * r];
    if (f >= tau[0]) gp[0] = fmax(gp[0], (double)sv + v0);
    if (f >= tau[1]) gp[1] = fmax(gp[1], (double)sv + v1);
  }
  double mm, gg;
  stage_gaps(tau[0], tau[1], gp[0], gp[1], &mm, &gg);
  const double sum_mm = wave_pairwise_sum(live ? mm : 0.0);
  const double sum_gp = wave_pairwise_sum(live ? gg : 0.0);
  if (lane == 0) {
    part_mm[tile * n_partial + chunk] = sum_mm;
    part_gp[tile * n_partial + chunk] = sum_gp;
  }
}

// Pairwise tree over n partials zero-padded to a power of two.  The stack
// holds one sum per set bit of the count so far: at most 15 for the largest
// count (2^20 samples / 64 per partial), so 16 entries, which the compiler
// keeps in registers.
__device__ __forceinline__ double partial_tree(const double *__restrict__ x, int64_t n) {
  double stack[16];
  int depth = 0;
  for (int64_t i = 0; i < n; ++i) {
    double v = x[i];
    for (int64_t m = i; m & 1; m >>= 1) v = stack[--depth] + v;
    stack[depth++] = v;
  }
  double sum = stack[depth - 1];
  for (int d = depth - 2; d >= 0; --d) sum = stack[d] + sum;
  return sum;
}

struct PickLex {
  double mm, gp;
  int tp, cell, e;  // e < 0: nothing
};

__device__ __forceinline__ bool better_lex(const PickLex &a, const PickLex &b) {
  if (a.e < 0) return false;
  if (b.e < 0) return true;
  if (a.mm != b.mm) return a.mm > b.mm;
  if (a.gp != b.gp) return a.gp > b.gp;
  if (a.tp != b.tp) return a.tp < b.tp;
  if (a.cell != b.cell) return a.cell < b.cell;
  return a.e < b.e;
}

// Scores of both stages and the lexicographic argmax: one wavefront per
// order, lanes over the candidates, then a shuffle reduction.  First the
// order's current gaps from its two certificate records (the max-min gap
// tau+ - tau-, the goodput gap |gp+ - gp-| / max(gp+, gp-), 0 when both are
// 0), written to gap_mm_out and gap_gp_out.
__global__ __launch_bounds__(64) void k_finalize_lex(DevProblem P, const CandInfo *__restrict__ info,
                                                     const uint8_t *__restrict__ measured, int32_t E, int32_t S,
                                                     const CertRec *__restrict__ rec,
                                                     double *__restrict__ gap_mm_out,
                                                     double *__restrict__ gap_gp_out,
                                                     const double *__restrict__ part_mm,
                                                     const double *__restrict__ part_gp, int64_t n_partial,
                                                     double *__restrict__ score_mm, double *__restrict__ score_gp,
                                                     int32_t *__restrict__ best) {
  const int o = blockIdx.x, lane = threadIdx.x;
  const CertRec *rm = rec + (size_t)o * 2, *rp = rm + 1;
  const double g_mm = (double)__int_as_float(rp->tau) - (double)__int_as_float(rm->tau);
  const double g64_m = rm->goodput64, g64_p = rp->goodput64;
  const double g_top = g64_p > g64_m ? g64_p : g64_m;
  const double g_gp = g_top > 0.0 ? fabs(g64_p - g64_m) / g_top : 0.0;
  if (lane == 0) {
    gap_mm_out[o] = g_mm;
    gap_gp_out[o] = g_gp;
  }
  PickLex mine{0.0, 0.0, 0, 0, -1};
  for (int e = lane; e < E; e += kWave) {
    const CandInfo ci = info[e];
    const size_t tile = (size_t)o * E + e;
    if (ci.cls < 0) {
      score_mm[tile] = score_gp[tile] = __builtin_nan("");
      continue;
    }
    if (measured[(size_t)o * P.N + ci.cell]) {
      score_mm[tile] = score_gp[tile] = 0.0;
      continue;
    }
    const double smm = g_mm - partial_tree(part_mm + tile * n_partial, n_partial) / (double)S;
    const double sgp = g_gp - partial_tree(part_gp + tile * n_partial, n_partial) / (double)S;
    score_mm[tile] = smm;
    score_gp[tile] = sgp;
    const PickLex c{smm, sgp, ci.tp, ci.cell, e};
    if (better_lex(c, mine)) mine = c;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    PickLex q;
    q.mm = __shfl_xor(mine.mm, off, kWave);
    q.gp = __shfl_xor(mine.gp, off, kWave);
    q.tp = __shfl_xor(mine.tp, off, kWave);
    q.cell = __shfl_xor(mine.cell, off, kWave);
    q.e = __shfl_xor(mine.e, off, kWave);
    if (better_lex(q, mine)) mine = q;
  }
  if (lane == 0 && best) best[o] = mine.e;
}

// ---------------------------------------------------------------------------
// Interval refit (Algorithm 1's fit step) under a structural prior: per
// class and load level, capacity per GPU is unimodal over the TP degrees in
// ascending order; per class and TP degree, the tail does not fall as the
// load level rises.  From the measured cells of the same row or column, an
// unmeasured cell gets
//   cap_lo >= t * min(max_{a < t measured} c_a / t_a, max_{z > t measured} c_z / t_z)
// (binary64, rounded down to binary32), and tail bounds from the nearest
// measured loads below and above; a bound that would empty the interval is
// dropped (the prior does not hold there).  One block per order, a thread
// per cell; measured cells are copied, or left alone when an output aliases
// its input (the refit reads only measured cells of other threads).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float round_down_f32(double x) {
  float v = (float)x;
  if ((double)v > x) v = nextafterf(v, -__builtin_inff());
  return v;
}

__global__ __launch_bounds__(256) void k_refit(DevProblem P, const float *__restrict__ cap_lo,
                                               const float *__restrict__ cap_hi, const float *__restrict__ tail_lo,
                                               const float *__restrict__ tail_hi,
                                               const uint8_t *__restrict__ measured, float *cap_lo_out,
                                               float *tail_lo_out, float *tail_hi_out) {
  const size_t off = (size_t)blockIdx.x * P.N;
  const int NT = P.NT, B = P.B;
  for (int c = threadIdx.x; c < P.N; c += blockDim.x) {
    if (measured[off + c]) {  // unchanged: copied unless refitting in place
      if (cap_lo_out != cap_lo) cap_lo_out[off + c] = cap_lo[off + c];
      if (tail_lo_out != tail_lo) tail_lo_out[off + c] = tail_lo[off + c];
      if (tail_hi_out != tail_hi) tail_hi_out[off + c] = tail_hi[off + c];
      continue;
    }
    const int b = c % B, t = (c / B) % NT, row = c - b - t * B;  // row: the class's first cell
    // capacity: best measured per-GPU value on each side of t at level b
    double left = -1.0, right = -1.0;
    for (int a = 0; a < NT; ++a) {
      const int ca = row + a * B + b;
      if (a == t || !measured[off + ca]) continue;
      const double q = (double)cap_lo[off + ca] / (double)P.tp[a];
      if (a < t) left = fmax(left, q);
      else right = fmax(right, q);
    }
    float lo = cap_lo[off + c];
    if (left >= 0.0 && right >= 0.0) lo = fmaxf(lo, round_down_f32((double)P.tp[t] * fmin(left, right)));
    if (lo <= cap_hi[off + c]) cap_lo_out[off + c] = lo;
    else if (cap_lo_out != cap_lo) cap_lo_out[off + c] = cap_lo[off + c];
    // tail: measured loads below bound it from below, above from above
    float tl = tail_lo[off + c], th = tail_hi[off + c];
    for (int b2 = 0; b2 < B; ++b2) {
      const int c2 = row + t * B + b2;
      if (b2 == b || !measured[off + c2]) continue;
      const float v = tail_lo[off + c2];
      if (b2 < b) tl = fmaxf(tl, v);
      else th = fminf(th, v);
    }
    if (tl <= th) {
      tail_lo_out[off + c] = tl;
      tail_hi_out[off + c] = th;
    } else {
      if (tail_lo_out != tail_lo) tail_lo_out[off + c] = tail_lo[off + c];
      if (tail_hi_out != tail_hi) tail_hi_out[off + c] = tail_hi[off + c];
    }
  }
}

// Samples of every (order, candidate) moved into the candidate's current
// intervals: min(max(x, lo), hi).  Block (run of 1024, tile).
__global__ __launch_bounds__(256) void k_clamp_samples(int32_t N, const int32_t *__restrict__ cand, int32_t E,
                                                       const float *__restrict__ cap_lo,
                                                       const float *__restrict__ cap_hi,
                                                       const float *__restrict__ tail_lo,
                                                       const float *__restrict__ tail_hi,
                                                       const float *__restrict__ cap_s,
                                                       const float *__restrict__ tail_s, int32_t S, uint32_t tiles,
                                                       float *__restrict__ cs_out, float *__restrict__ ts_out) {
  for (uint32_t tile = blockIdx.y; tile < tiles; tile += gridDim.y) {
    const uint32_t o = tile / (uint32_t)E, e = tile % (uint32_t)E;
    const int cell = cand[e];
    if (cell < 0 || cell >= N) continue;  // never scored
    const size_t ci = (size_t)o * N + cell;
    const float cl = cap_lo[ci], ch = cap_hi[ci], tl = tail_lo[ci], th = tail_hi[ci];
    const size_t base = (size_t)tile * S;
    for (int s = (int)blockIdx.x * 1024 + (int)threadIdx.x; s < S && s < ((int)blockIdx.x + 1) * 1024; s += 256) {
      cs_out[base + s] = fminf(fmaxf(cap_s[base + s], cl), ch);
      ts_out[base + s] = fminf(fmaxf(tail_s[base + s], tl), th);
    }
  }
}

// ---------------------------------------------------------------------------
// Profiling loop (Algorithm 1): per-trajectory bookkeeping between the
// certificate and scoring launches.
// ---------------------------------------------------------------------------
// Seconds one profiling cell runs (Section 5); a reveal costs this x TP.
constexpr double kCellSeconds = 300.0;

__global__ void k_loop_init(LoopDev L, int32_t O) {
  const int o = blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= O) return;
  L.running[o] = 1;
  L.state[o] = 0;
  L.finished[o] = 0;
  L.rounds[o] = 0;
  L.gpu_seconds[o] = 0.0;
  if (L.reveals)
    for (int j = 0; j < L.max_rounds; ++j) L.reveals[(size_t)o * L.max_rounds + j] = -1;
}

// One wavefront per trajectory: the lanes look at 64 candidates at a time.
__global__ __launch_bounds__(64) void k_loop_decide(DevProblem P, LoopDev L, const int32_t *__restrict__ cand,
                                                    int32_t E, int32_t O) {
  const int o = blockIdx.x, lane = threadIdx.x;
  if (!L.running[o]) return;
  const size_t off = (size_t)o * P.N;
  const int st = L.cert_state[o];
  if (lane == 0) {
    L.state[o] = st;
    L.fin.objective[o] = L.cons.objective[o];
    L.fin.floors_met[o] = L.cons.floors_met[o];
    L.fin.goodput[o] = L.cons.goodput[o];
  }
  for (int k = lane; k < P.K; k += kWave) {
    L.fin.tp_index[(size_t)o * P.K + k] = L.cons.tp_index[(size_t)o * P.K + k];
    L.fin.replicas[(size_t)o * P.K + k] = L.cons.replicas[(size_t)o * P.K + k];
  }
  bool end = st != 0;  // certified feasible or infeasible
  if (!end) {          // else: no unmeasured candidate left
    bool open = false;
    for (int e0 = 0; e0 < E && !open; e0 += kWave) {
      const int e = e0 + lane;
      const int c = e < E ? cand[e] : -1;
      open = __ballot(c >= 0 && c < P.N && !L.measured[off + c]) != 0;
    }
    end = !open;
  }
  if (!end) return;
  if (lane == 0) {
    L.finished[o] = 1;
    L.running[o] = 0;
  }
  for (int e = lane; e < E; e += kWave) {  // the scorer skips a finished trajectory
    const int c = cand[e];
    if (c >= 0 && c < P.N) L.measured[off + c] = 1;
  }
}

// Running trajectories, for the host's early-exit check.
__global__ __launch_bounds__(256) void k_loop_count(LoopDev L, int32_t O) {
  __shared__ int s_count[4];
  int count = 0;
  for (int o = threadIdx.x; o < O; o += blockDim.x) count += L.running[o] ? 1 : 0;
  count = wave_sum_int(count);
  if ((threadIdx.x & (kWave - 1)) == 0) s_count[threadIdx.x >> 6] = count;
  __syncthreads();
  if (threadIdx.x == 0) *L.n_running = s_count[0] + s_count[1] + s_count[2] + s_count[3];
}

// One wavefront per trajectory; under a fixed order the lanes look at 64
// entries of the order at a time and the first unmeasured one wins.
__global__ __launch_bounds__(64) void k_loop_reveal(DevProblem P, LoopDev L, const float *__restrict__ truth_cap,
                                                    const float *__restrict__ truth_tail,
                                                    const int32_t *__restrict__ cand, int32_t E, int32_t O,
                                                    int32_t policy, const int32_t *__restrict__ order) {
  const int o = blockIdx.x, lane = threadIdx.x;
  if (!L.running[o]) return;
  const size_t off = (size_t)o * P.N;
  int pick = -1;
  if (policy == 0) {
    pick = L.best[o];
  } else {
    for (int j0 = 0; j0 < E && pick < 0; j0 += kWave) {
      const int j = j0 + lane;
      const int e = j < E ? order[(size_t)o * E + j] : -1;
      const int c = (e >= 0 && e < E) ? cand[e] : -1;
      const uint64_t m = __ballot(c >= 0 && c < P.N && !L.measured[off + c]);
      if (m) pick = __shfl(e, __builtin_ctzll(m), kWave);
    }
  }
  if (lane != 0 || pick < 0 || pick >= E) return;
  const int cell = cand[pick];
  if (cell < 0 || cell >= P.N) return;
  L.cap_lo[off + cell] = L.cap_hi[off + cell] = truth_cap[off + cell];
  L.tail_lo[off + cell] = L.tail_hi[off + cell] = truth_tail[off + cell];
  L.measured[off + cell] = 1;
  L.gpu_seconds[o] += kCellSeconds * (double)P.tp[(cell / P.B) % P.NT];
  if (L.reveals && L.rounds[o] < L.max_rounds) L.reveals[(size_t)o * L.max_rounds + L.rounds[o]] = pick;
  L.rounds[o] += 1;
}

// Algorithm 1's last line, the best measured feasible allocation: the
// table of every trajectory with each unmeasured cell made infeasible (tail
// +inf, written over the working tail_lo, which the loop no longer needs);
// measured cells keep their point values.  The solve of (cap_lo, tail_lo)
// then serves only measured cells.
__global__ void k_loop_measured_table(LoopDev L, int64_t n) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  L.tail_lo[j] = L.measured[j] ? L.tail_hi[j] : __builtin_inff();
}

// The returned allocation: A- of a certified trajectory, the best measured
// feasible allocation (meas) of one that ended undecided; and its objective
// level (2) on the true table: the smallest fulfillment over the classes, an
// unserved class counting 0.
__global__ void k_loop_output(DevProblem P, LoopDev L, AllocOut meas, const int8_t *__restrict__ bmap,
                              const float *__restrict__ truth_cap, const float *__restrict__ truth_tail,
                              int32_t O, AllocOut out, float *__restrict__ tau_truth) {
  const int o = blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= O) return;
  const size_t off = (size_t)o * P.N;
  const AllocOut &A = L.state[o] == 0 ? meas : L.fin;
  if (out.objective) out.objective[o] = A.objective[o];
  if (out.floors_met) out.floors_met[o] = A.floors_met[o];
  if (out.goodput) out.goodput[o] = A.goodput[o];
  float v = __builtin_inff();
  bool unserved = false;
  for (int k = 0; k < P.K; ++k) {
    const int ti = A.tp_index[(size_t)o * P.K + k];
    const int r = A.replicas[(size_t)o * P.K + k];
    if (out.tp_index) out.tp_index[(size_t)o * P.K + k] = (uint8_t)ti;
    if (out.replicas) out.replicas[(size_t)o * P.K + k] = (uint16_t)r;
    if (r == 0) {
      unserved = true;
      continue;
    }
    const int cell = cell_of(P, k, ti, bmap[k * (P.G + 1) + r]);
    v = fminf(v, __int_as_float(ratio_bits(truth_cap[off + cell], truth_tail[off + cell], r, P.slo[k],
                                           P.rcp_demand[k])));
  }
  if (tau_truth) tau_truth[o] = unserved ? 0.0f : v;
}

// ---------------------------------------------------------------------------
// Class policies with several tail metrics and a success floor (Eq. 5 in
// full): each cell's (or sample's) metric vector becomes the single tail
// value the other kernels test against an SLO of 0.  Element-wise and bound
// by HBM: every block covers one row of cells or one run of a tile's
// samples, so the class -- and with it the limits, read from the kernel
// arguments at a uniform offset -- is known per block, and the hot loop does
// no integer division.
// ---------------------------------------------------------------------------
constexpr int kReduceThreads = 256;
constexpr int kReducePerThread = 4;  // samples per thread
constexpr int kReduceRun = kReduceThreads * kReducePerThread;

// Metric count: MC > 0 fixed at compile time, MC = 0 read from Q.M.
template <int MC>
__device__ __forceinline__ int policy_metrics(const DevPolicy &Q) {
  return MC > 0 ? MC : Q.M;
}

// Every metric of t within class k's limits (inclusive; NaN fails).  The
// tests are combined without short-circuit, so no branch splits the loads.
template <int MC>
__device__ __forceinline__ bool metrics_pass(const DevPolicy &Q, int k, const float *__restrict__ t) {
  const int M = policy_metrics<MC>(Q);
  bool ok = true;
#pragma unroll
  for (int m = 0; m < (MC > 0 ? MC : kMaxMetrics); ++m)
    if (MC > 0 || m < M) ok &= t[m] <= Q.limit[k * M + m];
  return ok;
}

// Cells: blockIdx.y walks the rows, blockIdx.x the 256-cell runs of a row.
template <int MC>
__global__ __launch_bounds__(kReduceThreads) void k_reduce_cells(DevPolicy Q, const float *__restrict__ tails,
                                                                 const float *__restrict__ success, int64_t rows,
                                                                 float *__restrict__ out) {
  const int M = policy_metrics<MC>(Q);
  const int c = (int)blockIdx.x * kReduceThreads + (int)threadIdx.x;
  if (c >= Q.N) return;
  const int k = c / Q.per_class;
  for (int64_t row = blockIdx.y; row < rows; row += gridDim.y) {
    const size_t j = (size_t)row * Q.N + c;
    bool ok = metrics_pass<MC>(Q, k, tails + j * M);
    if (Q.has_success) ok &= success[j] >= Q.success_min[k];
    out[j] = ok ? 0.0f : __builtin_inff();
  }
}

// Samples: blockIdx.y walks the (order, candidate) tiles, blockIdx.x the
// runs of kReduceRun samples of a tile; the class is that of the tile's
// candidate.  VEC (S a multiple of 4, arrays 16-byte aligned): a thread owns
// 4 consecutive samples and moves them with 16-byte loads and stores
// (M of them for the metrics, which are contiguous per sample).  Otherwise a
// thread takes samples threadIdx.x, + 256, + 512, + 768 of the run.
template <int MC, bool VEC>
__global__ __launch_bounds__(kReduceThreads) void k_reduce_samples(DevPolicy Q, const int32_t *__restrict__ cand,
                                                                   int32_t E, const float *__restrict__ tail_s,
                                                                   const float *__restrict__ succ_s, int32_t S,
                                                                   uint32_t tiles, float *__restrict__ out) {
  const int M = policy_metrics<MC>(Q);
  const float inf = __builtin_inff();
  for (uint32_t tile = blockIdx.y; tile < tiles; tile += gridDim.y) {
    const int cell = cand[tile % (uint32_t)E];
    const int k = (cell >= 0 && cell < Q.N) ? cell / Q.per_class : -1;
    const size_t base = (size_t)tile * S;
    if constexpr (VEC) {
      const int s = (int)blockIdx.x * kReduceRun + (int)threadIdx.x * kReducePerThread;
      if (s >= S) continue;  // S % 4 == 0: samples s .. s + 3 all exist
      float4 r = make_float4(inf, inf, inf, inf);
      if (k >= 0) {
        bool ok[kReducePerThread];
        // the success values first, so that their load is in flight with the metrics'
        float4 sc = make_float4(1.0f, 1.0f, 1.0f, 1.0f);
        float f = 0.0f;
        if (Q.has_success) {
          sc = *reinterpret_cast<const float4 *>(succ_s + base + s);
          f = Q.success_min[k];
        }
        if constexpr (MC > 0) {
          float t[kReducePerThread * MC], lim[MC];
          const float4 *src = reinterpret_cast<const float4 *>(tail_s + (base + s) * MC);
#pragma unroll
          for (int q = 0; q < MC; ++q) {
            const float4 v = src[q];
            t[4 * q + 0] = v.x; t[4 * q + 1] = v.y; t[4 * q + 2] = v.z; t[4 * q + 3] = v.w;
            lim[q] = Q.limit[k * MC + q];
          }
#pragma unroll
          for (int v = 0; v < kReducePerThread; ++v) {
            ok[v] = true;
#pragma unroll
            for (int m = 0; m < MC; ++m) ok[v] &= t[v * MC + m] <= lim[m];
          }
        } else {
#pragma unroll
          for (int v = 0; v < kReducePerThread; ++v) ok[v] = metrics_pass<0>(Q, k, tail_s + (base + s + v) * M);
        }
        if (Q.has_success) {
          ok[0] &= sc.x >= f; ok[1] &= sc.y >= f;
          ok[2] &= sc.z >= f; ok[3] &= sc.w >= f;
        }
        r = make_float4(ok[0] ? 0.0f : inf, ok[1] ? 0.0f : inf, ok[2] ? 0.0f : inf, ok[3] ? 0.0f : inf);
      }
      *reinterpret_cast<float4 *>(out + base + s) = r;
    } else {
#pragma unroll
      for (int v = 0; v < kReducePerThread; ++v) {
        const int s = (int)blockIdx.x * kReduceRun + v * kReduceThreads + (int)threadIdx.x;
        if (s >= S) break;
        bool ok = k >= 0;
        if (ok) ok = metrics_pass<0>(Q, k, tail_s + (base + s) * M);
        if (ok && Q.has_success) ok = succ_s[base + s] >= Q.success_min[k];
        out[base + s] = ok ? 0.0f : inf;
      }
    }
  }
}

__global__ void k_zero_flags(int32_t *__restrict__ flag) {
  if (threadIdx.x < 4) flag[threadIdx.x] = 0;
}

__global__ void k_validate_cands(const int32_t *__restrict__ cand, int32_t E, int32_t N,
                                 int32_t *__restrict__ flag) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e < E && (cand[e] < 0 || cand[e] >= N)) atomicAdd(&flag[1], 1);
}

__global__ void k_validate_cells(const float *__restrict__ cap, const float *__restrict__ tail,
                                 int64_t n, int32_t *__restrict__ flag) {
  int bad = 0;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const float c = cap[i], l = tail[i];
    const bool cap_ok = (c == 0.0f && !signbit(c)) ||
                        (c >= 0x1p-64f && c <= 0x1p64f);
    const bool tail_ok = !isnan(l) && l >= 0.0f;
    if (!cap_ok || !tail_ok) ++bad;
  }
  if (bad) atomicAdd(&flag[0], bad);
}

size_t lds_bytes_solver(const DevProblem &P, int n_alloc) {
  return sizeof(int) * (3 * (size_t)(P.G + 1) + (size_t)n_alloc * 2 * kMaxClasses);
}

}  // namespace

bool lane_kernel_supported(const DevProblem &P) {
  if (P.has_floor) return false;
  if (P.NT != 4 || P.tp[0] != 1 || P.tp[1] != 2 || P.tp[2] != 4 || P.tp[3] != 8) return false;
  return P.G == 16 || P.G == 32 || P.G == 64;
}

int lane_kernel_options(int G) { return G + G / 2 + G / 4 + G / 8; }

bool excl_kernel_supported(const DevProblem &P) { return !P.has_floor; }

// Workspace of fs_score_candidates_noalloc, for callers that cannot
// allocate: one copy per GPU the library runs on, held until the process
// ends, shared by every such call on that GPU.  Host code must not pass the
// name itself to a kernel (on the host it is a stand-in, not a device
// address): it uses the address scratch_address() returns, taken once per
// device when a context is created.
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

hipError_t scratch_address(void **ptr) { return hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch)); }

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Dynamic LDS the exclusion set-up kernel may request, and its block size
// (its passes are short and latency-bound: width shortens them).  Budgets
// of 512 GPUs and more take 1024 threads: the 16-class, G = 1024 scoring
// step took 94.7 us with 512 and 75.9 with 1024, the 8-class, G = 256 one
// 119.6 with 512 and 139.5 with 1024.
constexpr size_t kPrepLdsLimit = 60 * 1024;
constexpr int kPrepThreads = 512, kPrepThreadsWide = 1024, kPrepThreadsNarrow = 256, kPrepWideBudget = 512;

// LDS of the exclusion set-up besides its tables: cells (cap, tail), the
// class's cell maxima and replica ranges, and the load-level table.
static size_t prep_lds_small(const DevProblem &P) {
  const size_t KG = (size_t)P.K * P.G;
  return sizeof(int) * (2 * (size_t)P.N + 3 * (size_t)P.NT * P.B) + ((KG + 15) & ~(size_t)15);
}

// LDS of the set-up tables per block: B (K x G) and the two tree buffers.
static size_t prep_lds_tables(const DevProblem &P) {
  return sizeof(int) * (size_t)(P.K + prep_tree_a(P.K) + prep_tree_b(P.K)) * P.G;
}

// LDS of the general set-up's work-list block from staged inputs: counters,
// level ranges, candidates, revealed flags.
static size_t prep_list_lds(const DevProblem &P, int64_t O, int64_t E) {
  return 4 * (68 + 2 * (size_t)P.K * P.B + 2 * (size_t)E) + (size_t)O * P.N;
}

// Dynamic LDS of one general set-up block: a workgroup may hold 160 KiB on
// gfx950, less what the kernel declares statically.
constexpr size_t kPrepGeneralLdsLimit = 156 * 1024;

// LDS of the one-block-per-order set-up: the larger of a class block's and
// the work-list block's.
static size_t prep_order_lds(const DevProblem &P, int64_t O, int64_t E) {
  const size_t K = P.K, G = P.G, N = P.N, pc = (size_t)P.NT * P.B;
  const size_t nw = 2 * K <= 16 ? 2 * K : K;  // wavefronts with a per-wavefront area
  const size_t cls = 4 * (2 * N + 2 * K * G + (size_t)E + nw * 3 * pc) + ((N + 3) & ~(size_t)3) + K * G;
  const size_t lst = 4 * (68 + 2 * K * (size_t)P.B + 2 * (size_t)E) + (size_t)O * N;
  return cls > lst ? cls : lst;
}

static bool prep_order_fits(const DevProblem &P, int64_t O, int64_t E) {
  return P.G <= kPrepOrderMaxG && P.K <= kPrepOrderMaxK && prep_order_lds(P, O, E) <= kPrepLdsLimit;
}

// Options per (order, realisation): one per (class, TP, r).
static int32_t excl_thresholds(const DevProblem &P) {
  int per_class = 0;
  for (int t = 0; t < P.NT; ++t) per_class += P.G / P.tp[t];
  return P.K * per_class;
}

WsLayout ws_layout(const DevProblem &P, int64_t O, int64_t E, int64_t S) {
  WsLayout L{};
  size_t at = 0;
  L.bmap = at; at = align256(at + (size_t)P.K * (P.G + 1));
  L.cand = at; at = align256(at + sizeof(CandInfo) * (size_t)(E > 0 ? E : 1));
  L.base = at; at = align256(at + sizeof(int32_t) * 2 * (size_t)(O > 0 ? O : 1));
  L.pp = lane_kernel_supported(P) ? lane_kernel_options(P.G) : 0;
  L.opts = at; at = align256(at + sizeof(float) * 2 * (size_t)O * 2 * P.K * L.pp);
  L.n_partial = S > 0 ? (S + kWave - 1) / kWave : 1;
  L.partial = at; at = align256(at + sizeof(double) * (size_t)O * (size_t)E * L.n_partial);
  L.flag = at; at = align256(at + sizeof(int32_t) * 4);
  L.tiles = at; at = align256(at + sizeof(TileInfo) * (size_t)O * (size_t)E);
  const bool excl = excl_kernel_supported(P);
  // the exclusion set-up keeps B, P, S, H in LDS when they fit, else here
  const bool in_lds = prep_lds_small(P) + prep_lds_tables(P) <= kPrepGeneralLdsLimit;
  L.tabB = at;
  at = align256(at + (excl && !in_lds ? (size_t)O * 2 * P.K * 3 * sizeof(int) * P.K * P.G : 0));
  const size_t n_opt = excl ? (size_t)O * 2 * excl_thresholds(P) : 0;
  L.mopt = at; at = align256(at + sizeof(int32_t) * n_opt);
  L.thr = at; at = align256(at + sizeof(float) * n_opt);
  L.list = at; at = align256(at + sizeof(int4) * (size_t)O * (size_t)E);
  // B tables of the general set-up, one per (order, realisation, class)
  L.btab = at; at = align256(at + (excl ? sizeof(int32_t) * (size_t)O * 2 * P.K * P.G : 0));
  L.live = at; at = align256(at + sizeof(int32_t));
  L.crec = at; at = align256(at + sizeof(CertRec) * 2 * (size_t)(O > 0 ? O : 1));
  L.total = at;
  return L;
}

// Blocks of k_setup for the bucket map and for E candidate records.
static int setup_bucket_blocks(const DevProblem &P) {
  return (P.K * (P.G + 1) + kLexPrepThreads - 1) / kLexPrepThreads;
}
static int setup_cand_blocks(int32_t E) { return E > 0 ? (E + kLexPrepThreads - 1) / kLexPrepThreads : 0; }

hipError_t launch_setup(const DevProblem &P, const int32_t *cand, int32_t E, uint8_t *ws,
                        const WsLayout &L, hipStream_t s) {
  const int nb = setup_bucket_blocks(P), nc = setup_cand_blocks(E);
  k_setup<<<nb + nc, kLexPrepThreads, 0, s>>>(P, (int8_t *)(ws + L.bmap), nb, cand, E, (CandInfo *)(ws + L.cand), nc,
                                              nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr);
  return hipGetLastError();
}

// The exclusion scorer's set-up: per-order tables (U, M and thresholds of
// every option, base objectives, tile records) and the work list.
static hipError_t launch_excl_setup(const DevProblem &P, const ScoreArgs &a, hipStream_t s) {
  int32_t *base = (int32_t *)(a.ws + a.L.base);
  TileInfo *tiles = (TileInfo *)(a.ws + a.L.tiles);
  int32_t *mopt = (int32_t *)(a.ws + a.L.mopt);
  float *thr = (float *)(a.ws + a.L.thr);
  int4 *list = (int4 *)(a.ws + a.L.list);
  int32_t *live = (int32_t *)(a.ws + a.L.live);
  const int32_t n_thr = excl_thresholds(P);
  const int dump = a.tau_dump != nullptr;
  const size_t small = prep_lds_small(P), big = small + prep_lds_tables(P);
  if (a.setup == 0 && prep_order_fits(P, a.O, a.E)) {
    // the smallest level holding lambda / r; it falls as r grows, so one
    // pass over r per class moves it downwards only
    PrepLevels LV{};
    for (int k = 0; k < P.K; ++k) {
      int b = P.B;
      for (int r = 1; r <= P.G; ++r) {
        const float u = P.demand[k] / (float)r;
        while (b > 0 && !(P.levels[b - 1] < u)) --b;
        LV.lvl[k * kPrepOrderMaxG + r - 1] = (int8_t)(b < P.B ? b : -1);
      }
    }
    // compiled for the rank step's table count rounded up to 4, 8 or 16
    // and for at most 4 or 8 TP degrees (loops over them are unrolled)
#define FS_PREP_ORDER(KP, NTP)                                                                                    \
  k_prep_order<KP, NTP><<<2 * a.O + 1, prep_order_waves(P, a.O, a.E) * kWave, prep_order_lds(P, a.O, a.E), s>>>(    \
    P, a.cap_lo, a.cap_hi, a.tail_lo, a.tail_hi, a.measured, a.cand, a.E, a.O, dump, tiles, base, mopt, thr,  \
    n_thr, list, live, a.thr_search, LV)
#define FS_PREP_ORDER_K(NTP)                  \
  if (P.K <= 4) FS_PREP_ORDER(4, NTP);        \
  else if (P.K <= 8) FS_PREP_ORDER(8, NTP);   \
  else FS_PREP_ORDER(16, NTP);
    if (P.NT <= 4) {
      FS_PREP_ORDER_K(4)
    } else {
      FS_PREP_ORDER_K(8)
    }
#undef FS_PREP_ORDER_K
#undef FS_PREP_ORDER
  } else {
    // the work-list block reads staged inputs when they fit; tables in
    // LDS when they fit, else in the workspace
    const size_t lst = prep_list_lds(P, a.O, a.E);
    const int staged = lst <= kPrepGeneralLdsLimit;
    const bool in_lds = big <= kPrepGeneralLdsLimit;
    size_t lds = in_lds ? big : small;
    if (staged && lst > lds) lds = lst;
    int32_t *gtab = in_lds ? nullptr : (int32_t *)(a.ws + a.L.tabB);
    int32_t *btab = (int32_t *)(a.ws + a.L.btab);
    {
      const size_t blds = sizeof(int) * (size_t)P.G + 2 * sizeof(float) * (size_t)P.NT * P.B;
      const bool large = P.G >= kPrepWideBudget;
      const void *fn = large ? reinterpret_cast<const void *>(&k_prep_btab<kBtabThreadsLarge>)
                             : reinterpret_cast<const void *>(&k_prep_btab<kBtabThreadsSmall>);
      if (blds > 64 * 1024) {
        const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)blds);
        if (e != hipSuccess) return e;
      }
      if (large) {
        k_prep_btab<kBtabThreadsLarge><<<dim3(2, a.O, P.K), kBtabThreadsLarge, blds, s>>>(
            P, a.cap_lo, a.cap_hi, a.tail_lo, a.tail_hi, btab);
      } else {
        k_prep_btab<kBtabThreadsSmall><<<dim3(2, a.O, P.K), kBtabThreadsSmall, blds, s>>>(
            P, a.cap_lo, a.cap_hi, a.tail_lo, a.tail_hi, btab);
      }
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    const dim3 grid(2, a.O, P.K + 1);
#define FS_PREP_GENERAL(LDS, TH)                                                                                  \
  {                                                                                                               \
    if (lds > 64 * 1024) {                                                                                        \
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_prep<LDS, TH>),                  \
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);             \
      if (e != hipSuccess) return e;                                                                              \
    }                                                                                                             \
    k_prep<LDS, TH><<<grid, TH, lds, s>>>(P, a.cap_lo, a.cap_hi, a.tail_lo, a.tail_hi, a.measured, a.cand, a.E,   \
                                          dump, gtab, tiles, base, mopt, thr, n_thr, list, live, a.thr_search,    \
                                          staged, btab);                                                          \
  }
    // below a budget of 512: 256 threads per block once the class blocks
    // fill the GPU (more blocks resident at a time; 8 classes at G = 256
    // over 64 orders: step 80.5 -> 74 us; 128 threads: 82 us), else 512
    const bool narrow = (int64_t)2 * a.O * P.K >= 256;
    if (narrow && P.G < kPrepWideBudget) {
      if (in_lds) FS_PREP_GENERAL(true, kPrepThreadsNarrow)
      else FS_PREP_GENERAL(false, kPrepThreadsNarrow)
    } else if (P.G >= kPrepWideBudget) {
      if (in_lds) FS_PREP_GENERAL(true, kPrepThreadsWide)
      else FS_PREP_GENERAL(false, kPrepThreadsWide)
    } else {
      if (in_lds) FS_PREP_GENERAL(true, kPrepThreads)
      else FS_PREP_GENERAL(false, kPrepThreads)
    }
#undef FS_PREP_GENERAL
  }
  return hipGetLastError();
}

hipError_t launch_score(const DevProblem &P, const ScoreArgs &a, hipStream_t s) {
  const int8_t *bmap = (const int8_t *)(a.ws + a.L.bmap);
  CandInfo *info = (CandInfo *)(a.ws + a.L.cand);
  int32_t *base = (int32_t *)(a.ws + a.L.base);
  double *partial = (double *)(a.ws + a.L.partial);
  const size_t lds = lds_bytes_solver(P, 0);
  if (a.O == 0) return hipSuccess;
  if (a.kernel == 3) {
    constexpr int kSpl = 8;
    TileInfo *tiles = (TileInfo *)(a.ws + a.L.tiles);
    int32_t *mopt = (int32_t *)(a.ws + a.L.mopt);
    float *thr = (float *)(a.ws + a.L.thr);
    int4 *list = (int4 *)(a.ws + a.L.list);
    const int32_t n_thr = excl_thresholds(P);
    hipError_t es = launch_excl_setup(P, a, s);
    if (es != hipSuccess) return es;
    if (a.E == 0) {
      k_finalize<<<a.O, 64, 0, s>>>(P, info, a.measured, 0, a.S, base, partial, 1, a.score, a.gap_now,
                                    a.best);
      return hipGetLastError();
    }
    // Chunks of 1024 samples when the default grid would get more than 16
    // chunks of 512 per wavefront: on the 8-class, G = 256 workload (43
    // per wavefront) the scorer ran 33.0 us against 35.9 with 512; with
    // about 5 per wavefront (the 4-class, G = 64 one) 512 stays faster.
    const int64_t chunks512 = (int64_t)(a.S + 511) / 512 * a.O * a.E;
    const int spl = a.spl == 4 || a.spl == 8 || a.spl == 16 ? a.spl
                    : chunks512 > 16 * (int64_t)kScorerWaves ? 16 : kSpl;
    const int64_t chunk = 64 * spl;
    const int64_t n_partial = (a.S + chunk - 1) / chunk;
    // LDS: per-class constants, then M and thresholds of a range longer
    // than a wavefront (the longest range has G / tp[0] options)
    const int32_t range_max = P.G / P.tp[0];
    const size_t mlds = (size_t)P.K * (sizeof(double) + sizeof(float)) +
                        (range_max >= kWave ? 4 * sizeof(int) * (size_t)range_max : 0);
    const int64_t items = n_partial * a.O * a.E;  // upper bound of the live items
    const int64_t waves = a.waves > 0 ? a.waves : kScorerWaves;
    const unsigned grid = (unsigned)(items < waves ? items : waves);
    const int launches = a.ev_begin ? a.timing_launches : 1;
    if (a.ev_begin) (void)hipEventRecord(a.ev_begin, s);
    for (int rep = 0; rep < launches; ++rep) {
#define FS_EXCL_LAUNCH(SP, VEC, DUMP)                                                               \
  k_score_excl<SP, VEC, DUMP><<<grid, kWave, mlds, s>>>(P, tiles, mopt, thr, n_thr, list, a.cap_s,       \
                                                        a.tail_s, a.O, a.E, a.S, base, partial,     \
                                                        (int32_t)n_partial, a.tau_dump)
#define FS_EXCL_SPL(SP)                                         \
  if (a.tau_dump) {                                             \
    if (a.S % 4 == 0) FS_EXCL_LAUNCH(SP, true, true);           \
    else FS_EXCL_LAUNCH(SP, false, true);                       \
  } else {                                                      \
    if (a.S % 4 == 0) FS_EXCL_LAUNCH(SP, true, false);          \
    else FS_EXCL_LAUNCH(SP, false, false);                      \
  }
      if (spl == 16) { FS_EXCL_SPL(16) }
      else if (spl == 8) { FS_EXCL_SPL(8) }
      else { FS_EXCL_SPL(4) }
#undef FS_EXCL_SPL
#undef FS_EXCL_LAUNCH
    }
    if (a.ev_end) (void)hipEventRecord(a.ev_end, s);
    if (n_partial <= 16) {
      const int fw = (int)((a.E + 2 * kWave - 1) / (2 * kWave));
      const int nwf = fw < 1 ? 1 : (fw > kFinalizeMaxWaves ? kFinalizeMaxWaves : fw);
      k_finalize_excl<<<a.O, kWave * nwf, 0, s>>>(tiles, a.E, a.S, base, partial, n_partial, a.score,
                                                  a.gap_now, a.best);
    } else {
      k_tile_scores_wave<<<dim3((a.E + 3) / 4, a.O), 256, 0, s>>>(tiles, a.E, a.S, base, partial, n_partial,
                                                                 a.score);
      k_pick_best<<<a.O, 256, 0, s>>>(tiles, a.E, base, a.score, a.gap_now, a.best);
    }
    return hipGetLastError();
  }
  k_base<<<dim3(2, a.O), 64, lds, s>>>(P, bmap, a.cap_lo, a.cap_hi, a.tail_lo, a.tail_hi, base);
  int64_t n_partial = a.L.n_partial;
  const int launches = a.ev_begin ? a.timing_launches : 1;
  if (a.E > 0) {
    if (a.kernel == 2) {
      float *opts = (float *)(a.ws + a.L.opts);
      const dim3 grid((a.S + 255) / 256, a.E, a.O);
      n_partial = (a.S + 255) / 256;
#define FS_LANE_CASE(GG)                                                                         \
  case GG:                                                                                       \
    k_gather_options<GG><<<dim3(P.K, 2, a.O), 128, 0, s>>>(P, bmap, a.cap_lo, a.cap_hi,          \
                                                           a.tail_lo, a.tail_hi, opts);          \
    if (a.ev_begin) (void)hipEventRecord(a.ev_begin, s);                                         \
    for (int rep = 0; rep < launches; ++rep)                                                     \
      k_score_lane<GG><<<grid, 256, 0, s>>>(P, info, a.measured, opts, a.cap_s, a.tail_s, a.E,   \
                                            a.S, base, partial, n_partial, a.tau_dump);          \
    if (a.ev_end) (void)hipEventRecord(a.ev_end, s);                                             \
    break;
      switch (P.G) {
        FS_LANE_CASE(16)
        FS_LANE_CASE(32)
        FS_LANE_CASE(64)
        default:
          return hipErrorInvalidValue;
      }
#undef FS_LANE_CASE
    } else {
      const dim3 grid((a.S + kWave - 1) / kWave, a.E, a.O);
      if (a.ev_begin) (void)hipEventRecord(a.ev_begin, s);
      n_partial = (a.S + kWave - 1) / kWave;
      for (int rep = 0; rep < launches; ++rep)
        k_score_wave<<<grid, 64, lds, s>>>(P, bmap, info, a.cap_lo, a.cap_hi, a.tail_lo, a.tail_hi,
                                           a.measured, a.cap_s, a.tail_s, a.E, a.S, base, partial,
                                           n_partial, a.tau_dump);
      if (a.ev_end) (void)hipEventRecord(a.ev_end, s);
    }
  }
  k_finalize<<<a.O, 64, 0, s>>>(P, info, a.measured, a.E, a.S, base, partial, n_partial,
                                a.score, a.gap_now, a.best);
  return hipGetLastError();
}

hipError_t launch_solve_batch(const DevProblem &P, const float *cap, const float *tail, int64_t n,
                              AllocOut out, uint8_t *ws, const WsLayout &L, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const size_t base = lds_bytes_solver(P, 1), staged = base + stage_bytes(P);
  const int stage = stage_fits(staged) ? 1 : 0;
  if (stage)
    k_solve_dense<1><<<(unsigned)n, 64, staged, s>>>(P, (const int8_t *)(ws + L.bmap), cap, tail, n, out);
  else
    k_solve_dense<0><<<(unsigned)n, 64, base, s>>>(P, (const int8_t *)(ws + L.bmap), cap, tail, n, out);
  return hipGetLastError();
}

size_t lds_bytes_lex(const DevProblem &P, int n_alloc) {
  return sizeof(int) * (size_t)n_alloc * 2 * kMaxClasses + lex_work_bytes(P.K, P.G);
}

hipError_t launch_solve_batch_lex(const DevProblem &P, const float *cap, const float *tail, int64_t n,
                                  AllocOut out, double *gp64, uint8_t *ws, const WsLayout &L, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const size_t base = lds_bytes_lex(P, 1), staged = base + stage_bytes(P);
  const int stage = stage_fits(staged) ? 1 : 0;
  if (stage)
    k_solve_dense_lex<1><<<(unsigned)n, 64, staged, s>>>(P, (const int8_t *)(ws + L.bmap), cap, tail, n, out, gp64);
  else
    k_solve_dense_lex<0><<<(unsigned)n, 64, base, s>>>(P, (const int8_t *)(ws + L.bmap), cap, tail, n, out, gp64);
  return hipGetLastError();
}

hipError_t launch_certify_lex(const DevProblem &P, const float *cap_lo, const float *cap_hi, const float *tail_lo,
                              const float *tail_hi, const uint8_t *measured, int32_t O, float eps, int32_t *state,
                              AllocOut cons, AllocOut opt, double *gap_mm, double *gap_gp, uint8_t *ws,
                              const WsLayout &L, hipStream_t s, bool with_state) {
  if (O == 0) return hipSuccess;
  const size_t base = lds_bytes_lex(P, 1), staged = base + stage_bytes(P);
  const int stage = stage_fits(staged) ? 1 : 0;
  CertRec *rec = (CertRec *)(ws + L.crec);
  const int8_t *bmap = (const int8_t *)(ws + L.bmap);
  if (stage)
    k_certify_lex<1><<<dim3(2, O), 64, staged, s>>>(P, bmap, cap_lo, cap_hi, tail_lo, tail_hi, cons, opt, rec);
  else
    k_certify_lex<0><<<dim3(2, O), 64, base, s>>>(P, bmap, cap_lo, cap_hi, tail_lo, tail_hi, cons, opt, rec);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !with_state) return e;
  k_certify_state<<<O, 64, 0, s>>>(P, bmap, tail_hi, measured, eps, rec, 1, state, gap_mm, gap_gp);
  return hipGetLastError();
}

hipError_t launch_certify(const DevProblem &P, const float *cap_lo, const float *cap_hi,
                          const float *tail_lo, const float *tail_hi, const uint8_t *measured,
                          int32_t O, float eps, int32_t *state, AllocOut cons, AllocOut opt,
                          double *gap, uint8_t *ws, const WsLayout &L, hipStream_t s) {
  if (O == 0) return hipSuccess;
  const size_t base = lds_bytes_solver(P, 1), staged = base + stage_bytes(P);
  const int stage = stage_fits(staged) ? 1 : 0;
  CertRec *rec = (CertRec *)(ws + L.crec);
  const int8_t *bmap = (const int8_t *)(ws + L.bmap);
  if (stage)
    k_certify<1><<<dim3(2, O), 64, staged, s>>>(P, bmap, cap_lo, cap_hi, tail_lo, tail_hi, cons, opt, rec);
  else
    k_certify<0><<<dim3(2, O), 64, base, s>>>(P, bmap, cap_lo, cap_hi, tail_lo, tail_hi, cons, opt, rec);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_certify_state<<<O, 64, 0, s>>>(P, bmap, tail_hi, measured, eps, rec, 0, state, gap, nullptr);
  return hipGetLastError();
}

LoopLayout loop_layout(const DevProblem &P, int64_t O, int64_t E, int64_t S) {
  LoopLayout L{};
  L.score = ws_layout(P, O, E, S);
  size_t at = L.score.total;
  const size_t ON = (size_t)O * P.N, OK = (size_t)O * P.K;
  auto take = [&](size_t bytes) {
    const size_t here = at;
    at = align256(at + (bytes > 0 ? bytes : 1));
    return here;
  };
  L.cap_lo = take(4 * ON);
  L.cap_hi = take(4 * ON);
  L.tail_lo = take(4 * ON);
  L.tail_hi = take(4 * ON);
  L.measured = take(ON);
  L.cert_state = take(4 * (size_t)O);
  L.cons_obj = take(4 * (size_t)O);
  L.cons_tp = take(OK);
  L.cons_rep = take(2 * OK);
  L.cons_fm = take((size_t)O);
  L.cons_gp = take(4 * (size_t)O);
  L.fin_obj = take(4 * (size_t)O);
  L.fin_tp = take(OK);
  L.fin_rep = take(2 * OK);
  L.fin_fm = take((size_t)O);
  L.fin_gp = take(4 * (size_t)O);
  L.scores = take(8 * (size_t)O * (size_t)E);
  L.gap_now = take(8 * (size_t)O);
  L.best = take(4 * (size_t)O);
  L.running = take((size_t)O);
  L.n_running = take(4);
  L.scores_gp = take(8 * (size_t)O * (size_t)E);
  L.part_gp = take(8 * (size_t)O * (size_t)E * L.score.n_partial);
  L.gap_mm = take(8 * (size_t)O);
  L.gap_gp = take(8 * (size_t)O);
  L.lex_fast = lex_excl_regions(P, O, &at);
  L.total = at;
  return L;
}

RefitLayout refit_layout(const DevProblem &P, int64_t O, int64_t E, int64_t S, size_t start) {
  RefitLayout L{};
  size_t at = align256(start);
  auto take = [&](size_t bytes) {
    const size_t here = at;
    at = align256(at + (bytes > 0 ? bytes : 1));
    return here;
  };
  const size_t ON = (size_t)O * P.N, OES = (size_t)O * (size_t)E * (size_t)S;
  L.cap_lo = take(4 * ON);
  L.tail_lo = take(4 * ON);
  L.tail_hi = take(4 * ON);
  L.cap_s = take(4 * OES);
  L.tail_s = take(4 * OES);
  L.total = at;
  return L;
}

LoopDev loop_dev(const LoopLayout &L, uint8_t *ws, int64_t O) {
  (void)O;
  LoopDev d{};
  d.cap_lo = (float *)(ws + L.cap_lo);
  d.cap_hi = (float *)(ws + L.cap_hi);
  d.tail_lo = (float *)(ws + L.tail_lo);
  d.tail_hi = (float *)(ws + L.tail_hi);
  d.measured = ws + L.measured;
  d.cert_state = (int32_t *)(ws + L.cert_state);
  d.cons = AllocOut{(float *)(ws + L.cons_obj), ws + L.cons_tp, (uint16_t *)(ws + L.cons_rep), ws + L.cons_fm,
                    (float *)(ws + L.cons_gp)};
  d.fin = AllocOut{(float *)(ws + L.fin_obj), ws + L.fin_tp, (uint16_t *)(ws + L.fin_rep), ws + L.fin_fm,
                   (float *)(ws + L.fin_gp)};
  d.score = (double *)(ws + L.scores);
  d.gap_now = (double *)(ws + L.gap_now);
  d.best = (int32_t *)(ws + L.best);
  d.running = ws + L.running;
  d.n_running = (int32_t *)(ws + L.n_running);
  return d;
}

hipError_t launch_refit(const DevProblem &P, const float *cap_lo, const float *cap_hi, const float *tail_lo,
                        const float *tail_hi, const uint8_t *measured, int32_t O, float *cap_lo_out,
                        float *tail_lo_out, float *tail_hi_out, hipStream_t s) {
  if (O == 0) return hipSuccess;
  k_refit<<<O, 256, 0, s>>>(P, cap_lo, cap_hi, tail_lo, tail_hi, measured, cap_lo_out, tail_lo_out, tail_hi_out);
  return hipGetLastError();
}

hipError_t launch_clamp_samples(const DevProblem &P, const int32_t *cand, int32_t E, const float *cap_lo,
                                const float *cap_hi, const float *tail_lo, const float *tail_hi, const float *cap_s,
                                const float *tail_s, int32_t O, int32_t S, float *cs_out, float *ts_out,
                                hipStream_t s) {
  const uint32_t tiles = (uint32_t)O * (uint32_t)E;
  if (tiles == 0 || S == 0) return hipSuccess;
  const dim3 grid((unsigned)((S + 1023) / 1024), tiles < 65535 ? tiles : 65535u);
  k_clamp_samples<<<grid, 256, 0, s>>>(P.N, cand, E, cap_lo, cap_hi, tail_lo, tail_hi, cap_s, tail_s, S, tiles,
                                       cs_out, ts_out);
  return hipGetLastError();
}

LexExclRegions lex_excl_regions(const DevProblem &P, int64_t O, size_t *at) {
  LexExclRegions R{};
  const int PP = P.optoff[P.NT], nopt = P.K * PP;
  R.nbmax = nopt + 1;
  const size_t rows = (size_t)O * 2 * P.K * (size_t)(R.nbmax + 1);
  const size_t vbytes = sizeof(double) * rows * ((size_t)P.G + 1);
  R.fast = excl_kernel_supported(P) && lex_breaks_lds(nopt, P.N) <= kPrepGeneralLdsLimit &&
           lex_tables_lds(nopt, PP, P.G) <= kPrepGeneralLdsLimit &&
           lex_score_lds(R.nbmax, P.G / P.tp[0]) <= kPrepGeneralLdsLimit && vbytes <= ((size_t)4 << 30);
  auto take = [&](size_t bytes) {
    const size_t here = *at;
    *at = align256(*at + (bytes > 0 ? bytes : 1));
    return here;
  };
  if (!R.fast) return R;
  R.opt = take(sizeof(int2) * (size_t)O * 2 * nopt);
  R.bp = take(sizeof(float) * (size_t)O * 2 * R.nbmax);
  R.nbp = take(sizeof(int32_t) * (size_t)O * 2);
  R.V = take(vbytes);
  R.W = take(sizeof(double) * 4 * rows);
  return R;
}

LexScoreLayout lex_score_layout(const DevProblem &P, int64_t O, int64_t E, int64_t S) {
  LexScoreLayout L{};
  L.score = ws_layout(P, O, E, S);
  size_t at = L.score.total;
  auto take = [&](size_t bytes) {
    const size_t here = at;
    at = align256(at + (bytes > 0 ? bytes : 1));
    return here;
  };
  L.part_gp = take(sizeof(double) * (size_t)O * (size_t)E * L.score.n_partial);
  L.gap_mm = take(sizeof(double) * (size_t)O);
  L.gap_gp = take(sizeof(double) * (size_t)O);
  L.fast = lex_excl_regions(P, O, &at);
  L.total = at;
  return L;
}

hipError_t launch_score_lex(const DevProblem &P, const float *cap_lo, const float *cap_hi, const float *tail_lo,
                            const float *tail_hi, const uint8_t *measured, const int32_t *cand, const float *cap_s,
                            const float *tail_s, int32_t O, int32_t E, int32_t S, double *score_mm,
                            double *score_gp, double *gap_mm, double *gap_gp, int32_t *best, uint8_t *ws,
                            const LexScoreLayout &L, int fast, bool setup_here, hipStream_t s, hipStream_t side,
                            hipEvent_t fork, hipEvent_t join) {
  if (O == 0) return hipSuccess;
  double *gmm = gap_mm ? gap_mm : (double *)(ws + L.gap_mm);
  double *ggp = gap_gp ? gap_gp : (double *)(ws + L.gap_gp);
  const AllocOut none{nullptr, nullptr, nullptr, nullptr, nullptr};
  // One set-up launch (with setup_here the bucket map and the candidate
  // records; with the tables every order's option ratios and breakpoints),
  // then two chains.  The main stream builds the max-min stage's set-up (U, M
  // of every option), the goodput stage's tables and the scenarios; the
  // second stream, when there is one, solves the orders' own two
  // realisations (the certificate solves: a few wavefronts, bound by their
  // latency) into records, which the finalize turns into the current gaps.
  // The finalize waits for the second chain (join); a wait between streams
  // costs the host about as much as two launches.  The two chains write
  // disjoint workspace regions.  The main chain's set-up and tables are
  // enqueued first, so that they run while the host enqueues the rest.
  const bool par = side && fork && join;
  hipStream_t cs = par ? side : s;
  const bool tables = S > 0 && fast && L.fast.fast && E > 0;
  const LexExclRegions &X = L.fast;
  const int nopt = P.K * P.optoff[P.NT];
  hipError_t e = hipSuccess;
  {
    const int nb = setup_here ? setup_bucket_blocks(P) : 0, nc = setup_here ? setup_cand_blocks(E) : 0;
    const int nbr = tables ? 2 * O : 0;
    const size_t lds_b = nbr > 0 ? lex_breaks_lds(nopt, P.N) : 0;
    if (lds_b > 64 * 1024) {
      e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_setup), hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds_b);
      if (e != hipSuccess) return e;
    }
    if (nb + nc + nbr > 0) {
      k_setup<<<nb + nc + nbr, kLexPrepThreads, lds_b, s>>>(
          P, (int8_t *)(ws + L.score.bmap), nb, cand, E, (CandInfo *)(ws + L.score.cand), nc, cap_lo, cap_hi,
          tail_lo, tail_hi, X.nbmax, (int2 *)(ws + X.opt), (float *)(ws + X.bp), (int32_t *)(ws + X.nbp));
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  if (par) {
    e = hipEventRecord(fork, s);
    if (e != hipSuccess) return e;
  }
  if (tables) {
    ScoreArgs a{};
    a.cap_lo = cap_lo; a.cap_hi = cap_hi; a.tail_lo = tail_lo; a.tail_hi = tail_hi; a.measured = measured;
    a.cand = cand; a.cap_s = cap_s; a.tail_s = tail_s; a.O = O; a.E = E; a.S = S;
    a.ws = ws; a.L = L.score; a.kernel = 3;
    e = launch_excl_setup(P, a, s);
    if (e != hipSuccess) return e;
    const size_t lds_t = lex_tables_lds(nopt, P.optoff[P.NT], P.G);
    if (lds_t > 64 * 1024) {
      e = hipFuncSetAttribute(P.NT <= 4 ? reinterpret_cast<const void *>(&k_lex_tables<4>)
                                        : reinterpret_cast<const void *>(&k_lex_tables<8>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_t);
      if (e != hipSuccess) return e;
    }
    // blocks per (realisation, order, class): about kLexTableWaves
    // wavefronts in all, no more than the intervals can use
    const int64_t per = (int64_t)2 * O * P.K;
    const int64_t want = (kLexTableWaves / (per * (kLexPrepThreads / kWave))) + 1;
    const int64_t cap_split = (X.nbmax + 1 + kLexPrepThreads / kWave - 1) / (kLexPrepThreads / kWave);
    const int nsplit = (int)(want < cap_split ? want : cap_split);
    // compiled for at most 4 or 8 TP degrees (the loop over them is unrolled)
    if (P.NT <= 4) {
      k_lex_tables<4><<<dim3(2 * nsplit, O, P.K), kLexPrepThreads, lds_t, s>>>(
          P, (const int8_t *)(ws + L.score.bmap), (const int2 *)(ws + X.opt), (const float *)(ws + X.bp),
          (const int32_t *)(ws + X.nbp), X.nbmax, nsplit, (double *)(ws + X.V), (double *)(ws + X.W));
    } else {
      k_lex_tables<8><<<dim3(2 * nsplit, O, P.K), kLexPrepThreads, lds_t, s>>>(
          P, (const int8_t *)(ws + L.score.bmap), (const int2 *)(ws + X.opt), (const float *)(ws + X.bp),
          (const int32_t *)(ws + X.nbp), X.nbmax, nsplit, (double *)(ws + X.V), (double *)(ws + X.W));
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // the second chain: the certificate records only (the finalize forms the gaps)
  if (par) {
    e = hipStreamWaitEvent(side, fork, 0);
    if (e != hipSuccess) return e;
  }
  e = launch_certify_lex(P, cap_lo, cap_hi, tail_lo, tail_hi, measured, O, 0.0f, nullptr, none,
                         none, gmm, ggp, ws, L.score, cs, false);
  if (e != hipSuccess) return e;
  if (par) {
    e = hipEventRecord(join, side);
    if (e != hipSuccess) return e;
  }
  const int64_t n_partial = L.score.n_partial;
  double *pmm = (double *)(ws + L.score.partial), *pgp = (double *)(ws + L.part_gp);
  const CandInfo *info = (const CandInfo *)(ws + L.score.cand);
  if (tables) {
    const dim3 grid((unsigned)((S + kWave - 1) / kWave), (unsigned)E, (unsigned)O);
    const int32_t rmax = P.G / P.tp[0];  // the longest replica range
    const size_t lds_s = lex_score_lds(X.nbmax, rmax);
    if (lds_s > 64 * 1024) {
      e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_score_lex_excl),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_s);
      if (e != hipSuccess) return e;
    }
    k_score_lex_excl<<<grid, kWave, lds_s, s>>>(
        P, (const TileInfo *)(ws + L.score.tiles), (const int32_t *)(ws + L.score.mopt), excl_thresholds(P), cap_s,
        tail_s, E, S, (const float *)(ws + X.bp), (const int32_t *)(ws + X.nbp), X.nbmax, rmax,
        (const double *)(ws + X.V), (const double *)(ws + X.W), pmm, pgp, n_partial);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  } else if (S > 0 && E > 0) {
    const size_t base = lds_bytes_lex(P, 1), staged = base + stage2_bytes(P);
    const int stage = stage_fits(staged) ? 1 : 0;
    const dim3 grid((unsigned)((S + kWave - 1) / kWave), (unsigned)E, (unsigned)O);
    if (stage)
      k_score_lex_wave<1><<<grid, 64, staged, s>>>(P, (const int8_t *)(ws + L.score.bmap), info, cap_lo, cap_hi,
          tail_lo, tail_hi, measured, cap_s, tail_s, E, S, pmm, pgp, n_partial);
    else
      k_score_lex_wave<0><<<grid, 64, base, s>>>(P, (const int8_t *)(ws + L.score.bmap), info, cap_lo, cap_hi,
          tail_lo, tail_hi, measured, cap_s, tail_s, E, S, pmm, pgp, n_partial);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (par) {
    e = hipStreamWaitEvent(s, join, 0);
    if (e != hipSuccess) return e;
  }
  // with no candidates only the gaps are written (best stays as it was)
  k_finalize_lex<<<O, 64, 0, s>>>(P, info, measured, E, S, (const CertRec *)(ws + L.score.crec), gmm, ggp, pmm,
                                  pgp, S > 0 ? n_partial : 0, score_mm, score_gp, E > 0 ? best : nullptr);
  return hipGetLastError();
}

hipError_t launch_loop_init(const LoopDev &L, int32_t O, hipStream_t s) {
  if (O == 0) return hipSuccess;
  k_loop_init<<<(O + 255) / 256, 256, 0, s>>>(L, O);
  return hipGetLastError();
}

hipError_t launch_loop_decide(const DevProblem &P, const LoopDev &L, const int32_t *cand, int32_t E,
                              int32_t O, hipStream_t s) {
  if (O == 0) return hipSuccess;
  k_loop_decide<<<O, kWave, 0, s>>>(P, L, cand, E, O);
  return hipGetLastError();
}

hipError_t launch_loop_count(const LoopDev &L, int32_t O, hipStream_t s) {
  k_loop_count<<<1, 256, 0, s>>>(L, O);
  return hipGetLastError();
}

hipError_t launch_loop_reveal(const DevProblem &P, const LoopDev &L, const float *truth_cap,
                              const float *truth_tail, const int32_t *cand, int32_t E, int32_t O,
                              int32_t policy, const int32_t *order, hipStream_t s) {
  if (O == 0) return hipSuccess;
  k_loop_reveal<<<O, kWave, 0, s>>>(P, L, truth_cap, truth_tail, cand, E, O, policy, order);
  return hipGetLastError();
}

hipError_t launch_loop_measured_table(const DevProblem &P, const LoopDev &L, int32_t O, hipStream_t s) {
  const int64_t n = (int64_t)O * P.N;
  if (n == 0) return hipSuccess;
  k_loop_measured_table<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(L, n);
  return hipGetLastError();
}

hipError_t launch_loop_output(const DevProblem &P, const LoopDev &L, const AllocOut &meas, const uint8_t *ws,
                              const WsLayout &SL, const float *truth_cap, const float *truth_tail, int32_t O,
                              AllocOut out, float *tau_truth, hipStream_t s) {
  if (O == 0) return hipSuccess;
  k_loop_output<<<(O + 63) / 64, 64, 0, s>>>(P, L, meas, (const int8_t *)(ws + SL.bmap), truth_cap, truth_tail, O,
                                             out, tau_truth);
  return hipGetLastError();
}

hipError_t launch_reduce_cells(const DevPolicy &Q, const float *tails, const float *success, int64_t rows,
                               float *out, hipStream_t s) {
  if (rows == 0 || Q.N == 0) return hipSuccess;
  const dim3 grid((unsigned)((Q.N + kReduceThreads - 1) / kReduceThreads),
                  (unsigned)(rows < 65535 ? rows : 65535));
  switch (Q.M) {
    case 1: k_reduce_cells<1><<<grid, kReduceThreads, 0, s>>>(Q, tails, success, rows, out); break;
    case 2: k_reduce_cells<2><<<grid, kReduceThreads, 0, s>>>(Q, tails, success, rows, out); break;
    case 3: k_reduce_cells<3><<<grid, kReduceThreads, 0, s>>>(Q, tails, success, rows, out); break;
    case 4: k_reduce_cells<4><<<grid, kReduceThreads, 0, s>>>(Q, tails, success, rows, out); break;
    default: k_reduce_cells<0><<<grid, kReduceThreads, 0, s>>>(Q, tails, success, rows, out); break;
  }
  return hipGetLastError();
}

hipError_t launch_reduce_samples(const DevPolicy &Q, const int32_t *cand, int32_t E, const float *tail_s,
                                 const float *succ_s, int32_t O, int32_t S, float *out, hipStream_t s) {
  const uint32_t tiles = (uint32_t)O * (uint32_t)E;  // O, E <= 65535
  if (tiles == 0 || S == 0) return hipSuccess;
  const dim3 grid((unsigned)((S + kReduceRun - 1) / kReduceRun), tiles < 65535 ? tiles : 65535u);
  auto aligned = [](const void *q) { return ((uintptr_t)q & 15) == 0; };
  const bool vec = S % 4 == 0 && aligned(tail_s) && aligned(out) && (!Q.has_success || aligned(succ_s));
#define FS_RED_S(MC, V) k_reduce_samples<MC, V><<<grid, kReduceThreads, 0, s>>>(Q, cand, E, tail_s, succ_s, S, tiles, out)
  if (!vec) {
    FS_RED_S(0, false);
  } else {
    switch (Q.M) {
      case 1: FS_RED_S(1, true); break;
      case 2: FS_RED_S(2, true); break;
      case 3: FS_RED_S(3, true); break;
      case 4: FS_RED_S(4, true); break;
      default: FS_RED_S(0, true); break;
    }
  }
#undef FS_RED_S
  return hipGetLastError();
}

hipError_t launch_zero_flags(int32_t *flag, hipStream_t s) {
  k_zero_flags<<<1, 64, 0, s>>>(flag);
  return hipGetLastError();
}

hipError_t launch_validate_cands(const int32_t *cand, int32_t E, int32_t N, int32_t *flag, hipStream_t s) {
  if (E == 0) return hipSuccess;
  k_validate_cands<<<(E + 255) / 256, 256, 0, s>>>(cand, E, N, flag);
  return hipGetLastError();
}

hipError_t launch_validate_cells(const float *cap, const float *tail, int64_t n, int32_t *flag,
                                 hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096;
  k_validate_cells<<<(unsigned)blocks, 256, 0, s>>>(cap, tail, n, flag);
  return hipGetLastError();
}

}  // namespace fs
