"""Seeded synthetic workloads shaped like FleetSieve's evaluation.

This module only draws inputs; it holds none of the method's arithmetic (no
fulfillment, no solve, no score).  Both the HIP path and the CPU oracle are fed
from it.  The paper's measurement grid (H100 cells of a 31B FP8 model under
Azure conversation/code traces, Section 5) is not available; these inputs
stand in for it with the same structure:

* workload classes with a demand lambda_i and a tail SLO L_i (Section 3);
* TP degrees including {2, 4, 8} and a geometric per-replica load ladder
  (Section 5: loads are ordinal rungs of an arrival-scale ladder);
* per-GPU capacity c/t with an interior knee at TP4 (Table 1, Fig. 1a);
* a completion-tail that grows with load and shrinks with TP, so a heavy
  load can make TP4 infeasible while TP8 stays feasible (Fig. 1b);
* capacity and tail intervals per cell (Section 4.1), partially collapsed to
  a hidden truth along random reveal orders (Section 5, "200 random reveal
  orders"), with capacities on a 1/64 req/s grid;
* outcome samples drawn uniformly inside each candidate's intervals: the
  capacity on the 1/64 grid, the tail in binary32.

Cell layout: cell(i, t, b) = (i * n_tp + t) * n_levels + b.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

QUANTUM = 1.0 / 64.0  # capacity grid, req/s

# Tail-median factor per TP degree: larger TP shortens the completion tail.
TAIL_TP_FACTOR = {1: 1.3, 2: 1.15, 4: 1.0, 8: 0.5, 16: 0.4}
SLO_CHOICES = (1.0, 2.0, 5.0, 30.0, 120.0, 600.0)


@dataclass
class Problem:
    """The allocation problem of Section 3 (host arrays)."""
    tp: np.ndarray          # [n_tp] int32, ascending GPUs per replica
    levels: np.ndarray      # [n_levels] float32, ascending per-replica req/s
    demand: np.ndarray      # [K] float32 lambda_i
    slo: np.ndarray         # [K] float32 L_i
    budget: int             # G
    floor_rps: np.ndarray | None = None  # [K] float32, 0 = not critical

    def __post_init__(self):
        self.tp = np.ascontiguousarray(self.tp, dtype=np.int32)
        self.levels = np.ascontiguousarray(self.levels, dtype=np.float32)
        self.demand = np.ascontiguousarray(self.demand, dtype=np.float32)
        self.slo = np.ascontiguousarray(self.slo, dtype=np.float32)
        if self.floor_rps is not None:
            self.floor_rps = np.ascontiguousarray(self.floor_rps, dtype=np.float32)
        self.budget = int(self.budget)

    @property
    def n_classes(self) -> int:
        return len(self.demand)

    @property
    def n_tp(self) -> int:
        return len(self.tp)

    @property
    def n_levels(self) -> int:
        return len(self.levels)

    @property
    def n_cells(self) -> int:
        return self.n_classes * self.n_tp * self.n_levels

    def cell(self, i: int, t: int, b: int) -> int:
        return (i * self.n_tp + t) * self.n_levels + b

    def cell_coords(self, cell: int) -> tuple:
        b = cell % self.n_levels
        t = (cell // self.n_levels) % self.n_tp
        i = cell // (self.n_levels * self.n_tp)
        return i, t, b


@dataclass
class Intervals:
    """Per-order capacity and tail intervals (Section 4.1), [O][N]."""
    cap_lo: np.ndarray
    cap_hi: np.ndarray
    tail_lo: np.ndarray
    tail_hi: np.ndarray
    measured: np.ndarray  # uint8

    @property
    def n_orders(self) -> int:
        return self.cap_lo.shape[0]

    def subset(self, orders) -> "Intervals":
        idx = np.asarray(orders)
        return Intervals(self.cap_lo[idx], self.cap_hi[idx], self.tail_lo[idx], self.tail_hi[idx],
                         self.measured[idx])


@dataclass
class Workload:
    name: str
    seed: int
    problem: Problem
    intervals: Intervals          # [O][N]
    cand: np.ndarray              # [E] int32 cell indices
    cap_s: np.ndarray | None      # [O][E][S] float32
    tail_s: np.ndarray | None     # [O][E][S] float32
    truth_cap: np.ndarray         # [N] hidden truth used for reveals
    truth_tail: np.ndarray
    orders: np.ndarray            # which of the workload's reveal orders these are
    n_samples: int
    recipe: dict = field(default_factory=dict)

    @property
    def n_orders(self) -> int:
        return self.intervals.n_orders

    @property
    def n_cand(self) -> int:
        return len(self.cand)


def _geometric(start: float, n: int) -> list:
    return [start * (2.0 ** k) for k in range(n)]


# The seeded synthetic workloads, by name.  Each has its own seed.
WORKLOADS = {
    "tiny-2class-G16": dict(seed=1000, K=2, tp=[1, 2, 4, 8], G=16, levels=[0.5, 1.0, 2.0],
            demand=("fixed", [4.0, 2.0]), slo=("fixed", [30.0, 30.0]),
            cap_range=(0.2, 3.0), cap_width=(0.05, 0.3), tail_sigma=0.4, tail_alpha=1.0,
            tail_tp_factor=False, tail_width=(0.1, 0.4), orders=1, reveal=False,
            cand=("subset", 8), samples=64),
    "paper-shaped-2class-G16": dict(seed=1001, K=2, tp=[1, 2, 4, 8], G=16,
            levels=[0.25, 0.5, 1.0, 2.0, 4.0, 8.0],
            # code at 3 req/s (not 2) so the 16-GPU budget binds and decision
            # gaps stay open; at 4 / 2 req/s every realisation serves both fully
            demand=("fixed", [4.0, 3.0]), slo=("fixed", [30.0, 30.0]),
            cap_range=(0.2, 3.0), cap_width=(0.05, 0.3), tail_sigma=0.4, tail_alpha=1.5,
            tail_tp_factor=True, tail_width=(0.1, 0.4), orders=200, reveal=True,
            cand=("all",), samples=1024),
    "4class-G64": dict(seed=1002, K=4, tp=[1, 2, 4, 8], G=64, levels=_geometric(0.125, 8),
            demand=("uniform", 1.0, 20.0), slo=("fixed", [30.0, 20.0, 2.0, 300.0]),
            cap_range=(0.1, 5.0), cap_width=(0.05, 0.3), tail_sigma=0.5, tail_alpha=1.0,
            tail_tp_factor=True, tail_width=(0.1, 0.4), orders=16, reveal=True,
            cand=("all",), samples=4096),
    "8class-G256": dict(seed=1003, K=8, tp=[1, 2, 4, 8], G=256, levels=_geometric(0.125, 8),
            demand=("uniform", 0.5, 50.0), slo=("choice", SLO_CHOICES),
            cap_range=(0.1, 5.0), cap_width=(0.02, 0.5), tail_sigma=0.5, tail_alpha=1.0,
            tail_tp_factor=True, tail_width=(0.02, 0.5), orders=64, reveal=True,
            cand=("all",), samples=4096),
    "16class-G1024": dict(seed=1004, K=16, tp=[1, 2, 4, 8, 16], G=1024, levels=_geometric(0.0625, 12),
            demand=("uniform", 1.0, 200.0), slo=("choice", SLO_CHOICES),
            cap_range=(0.1, 5.0), cap_width=(0.02, 0.5), tail_sigma=0.5, tail_alpha=1.0,
            tail_tp_factor=True, tail_width=(0.02, 0.5), orders=4, reveal=True,
            cand=("all",), samples=256),
    # Class counts between the two- and four-class shapes and the 16-class
    # fleet at budgets of one wavefront or less: they exercise the set-up's
    # wavefront layouts (two wavefronts per class up to 8 classes, one per
    # class up to 16).
    "6class-G32": dict(seed=1007, K=6, tp=[1, 2, 4, 8], G=32, levels=_geometric(0.125, 8),
            demand=("uniform", 0.5, 3.0), slo=("choice", SLO_CHOICES),
            cap_range=(0.1, 5.0), cap_width=(0.05, 0.3), tail_sigma=0.5, tail_alpha=1.0,
            tail_tp_factor=True, tail_width=(0.1, 0.4), orders=8, reveal=True,
            cand=("all",), samples=512),
    "12class-G64": dict(seed=1008, K=12, tp=[1, 2, 4, 8], G=64, levels=_geometric(0.125, 8),
            demand=("uniform", 1.0, 8.0), slo=("choice", SLO_CHOICES),
            cap_range=(0.1, 5.0), cap_width=(0.05, 0.3), tail_sigma=0.5, tail_alpha=1.0,
            tail_tp_factor=True, tail_width=(0.1, 0.4), orders=4, reveal=True,
            cand=("all",), samples=256),
    # Truth drawn first with the structure the interval refit assumes
    # (capacity per GPU unimodal over TP with its knee at TP4, tail
    # nondecreasing in the load), intervals around it.
    "paper-shaped-2class-G16-knee": dict(seed=1005, K=2, tp=[1, 2, 4, 8], G=16,
            levels=[0.25, 0.5, 1.0, 2.0, 4.0, 8.0], demand=("fixed", [4.0, 3.0]), slo=("fixed", [30.0, 30.0]),
            cap_range=(0.2, 3.0), cap_width=(0.05, 0.3), tail_sigma=0.4, tail_alpha=1.5,
            tail_tp_factor=True, tail_width=(0.1, 0.4), orders=200, reveal=True,
            cand=("all",), samples=1024, structure=True),
    "4class-G64-knee": dict(seed=1006, K=4, tp=[1, 2, 4, 8], G=64, levels=_geometric(0.125, 8),
            demand=("uniform", 1.0, 20.0), slo=("fixed", [30.0, 20.0, 2.0, 300.0]),
            cap_range=(0.1, 5.0), cap_width=(0.05, 0.3), tail_sigma=0.5, tail_alpha=1.0,
            tail_tp_factor=True, tail_width=(0.1, 0.4), orders=16, reveal=True,
            cand=("all",), samples=4096, structure=True),
}


def q64(x):
    """Round to the nearest multiple of 1/64 req/s, at least 1/64."""
    return np.maximum(np.rint(np.asarray(x, dtype=np.float64) * 64.0), 1.0) / 64.0


def _knee_capacities(rng, tp, lo, hi, max_tries=10000):
    """|T| per-replica capacities, quantised, with per-GPU capacity c/t
    strictly largest at TP4 (the interior knee of Table 1)."""
    tp = np.asarray(tp)
    has4 = 4 in tp.tolist()
    k4 = tp.tolist().index(4) if has4 else None
    for _ in range(max_tries):
        c = q64(rng.uniform(lo, hi, size=len(tp)))
        if not has4:
            return c
        per_gpu = c / tp
        others = np.delete(per_gpu, k4)
        if np.all(per_gpu[k4] > others):
            return c
    raise RuntimeError("capacity draw could not place the knee at TP4")


def _problem_for(name: str, rng) -> Problem:
    c = WORKLOADS[name]
    K = c["K"]
    kind = c["demand"][0]
    if kind == "fixed":
        demand = np.array(c["demand"][1], dtype=np.float64)
    else:
        demand = rng.uniform(c["demand"][1], c["demand"][2], size=K)
    kind = c["slo"][0]
    if kind == "fixed":
        slo = np.array(c["slo"][1], dtype=np.float64)
    else:
        slo = rng.choice(np.array(c["slo"][1]), size=K)
    return Problem(tp=c["tp"], levels=c["levels"], demand=demand.astype(np.float32),
                   slo=slo.astype(np.float32), budget=c["G"], floor_rps=None)


def _initial_intervals(name: str, problem: Problem, rng):
    """Initial interval per cell: [c_lo, c_hi] and [l_lo, l_hi], float64."""
    c = WORKLOADS[name]
    K, T, B = problem.n_classes, problem.n_tp, problem.n_levels
    N = problem.n_cells
    cap_lo = np.zeros(N)
    cap_hi = np.zeros(N)
    tail_lo = np.zeros(N)
    tail_hi = np.zeros(N)
    for i in range(K):
        for b in range(B):
            caps = _knee_capacities(rng, problem.tp, *c["cap_range"])
            for t in range(T):
                cell = problem.cell(i, t, b)
                w = rng.uniform(*c["cap_width"])
                cap_lo[cell] = caps[t]
                cap_hi[cell] = max(q64(caps[t] * (1.0 + w)), caps[t])
    for i in range(K):
        for t in range(T):
            rho = TAIL_TP_FACTOR[int(problem.tp[t])] if c["tail_tp_factor"] else 1.0
            for b in range(B):
                cell = problem.cell(i, t, b)
                load = float(problem.levels[b])
                median = (float(problem.slo[i]) / 3.0) * (1.0 + load) ** c["tail_alpha"] * rho
                lo = np.float32(median * np.exp(c["tail_sigma"] * rng.standard_normal()))
                hi = np.float32(float(lo) * (1.0 + rng.uniform(*c["tail_width"])))
                tail_lo[cell] = lo
                tail_hi[cell] = max(hi, lo)
    return cap_lo, cap_hi, tail_lo, tail_hi


def _structured_truth(name: str, problem: Problem, rng):
    """Truth with the refit's structure, then intervals containing it.
    Per (class, level): capacity per GPU at the knee (TP4) drawn from the
    workload's range over 4, each step away from the knee keeping a factor
    U[0.55, 0.95] of its neighbour; per-replica values on the 1/64 grid
    (redrawn until the per-GPU values stay unimodal after rounding).  Per
    (class, TP): tails as in the generic workloads, then a running maximum
    over increasing load.  Intervals: capacity [q64(c (1 - w)), q64(c (1 +
    w'))] and tail [l / (1 + u), l (1 + u')], w, w', u, u' from the widths."""
    c = WORKLOADS[name]
    K, T, B = problem.n_classes, problem.n_tp, problem.n_levels
    N = problem.n_cells
    tp = [int(x) for x in problem.tp]
    knee = tp.index(4)
    truth_cap = np.zeros(N)
    truth_tail = np.zeros(N, np.float32)
    for i in range(K):
        for b in range(B):
            while True:
                g = np.zeros(T)
                g[knee] = rng.uniform(*c["cap_range"]) / 4.0
                for t in range(knee - 1, -1, -1):
                    g[t] = g[t + 1] * rng.uniform(0.55, 0.95)
                for t in range(knee + 1, T):
                    g[t] = g[t - 1] * rng.uniform(0.55, 0.95)
                caps = q64(g * np.array(tp, float))
                per_gpu = caps / np.array(tp, float)
                if np.all(np.diff(per_gpu[:knee + 1]) >= 0) and np.all(np.diff(per_gpu[knee:]) <= 0):
                    break
            for t in range(T):
                truth_cap[problem.cell(i, t, b)] = caps[t]
    for i in range(K):
        for t in range(T):
            rho = TAIL_TP_FACTOR[int(problem.tp[t])] if c["tail_tp_factor"] else 1.0
            run = np.float32(0.0)
            for b in range(B):
                load = float(problem.levels[b])
                median = (float(problem.slo[i]) / 3.0) * (1.0 + load) ** c["tail_alpha"] * rho
                run = max(run, np.float32(median * np.exp(c["tail_sigma"] * rng.standard_normal())))
                truth_tail[problem.cell(i, t, b)] = run
    w_lo = rng.uniform(*c["cap_width"], size=N)
    w_hi = rng.uniform(*c["cap_width"], size=N)
    cap_lo = np.minimum(q64(truth_cap * (1.0 - w_lo)), truth_cap)
    cap_hi = np.maximum(q64(truth_cap * (1.0 + w_hi)), truth_cap)
    u_lo = rng.uniform(*c["tail_width"], size=N)
    u_hi = rng.uniform(*c["tail_width"], size=N)
    tail_lo = np.minimum((truth_tail / (1.0 + u_lo)).astype(np.float32), truth_tail)
    tail_hi = np.maximum((truth_tail * (1.0 + u_hi)).astype(np.float32), truth_tail)
    return (cap_lo, cap_hi, tail_lo.astype(np.float64), tail_hi.astype(np.float64),
            truth_cap.astype(np.float32), truth_tail)


def _draw_inside(rng, cap_lo, cap_hi, tail_lo, tail_hi, shape=None):
    """Uniform draw inside intervals: capacity on the 1/64 grid, tail fp32."""
    steps = np.rint((np.asarray(cap_hi) - np.asarray(cap_lo)) * 64.0).astype(np.int64)
    if shape is None:
        k = rng.integers(0, steps + 1)
        u = rng.random(np.shape(cap_lo))
    else:
        k = rng.integers(0, steps[..., None] + 1, size=shape)
        u = rng.random(shape)
        cap_lo, tail_lo, tail_hi = (np.asarray(a)[..., None] for a in (cap_lo, tail_lo, tail_hi))
    cap = (np.rint(np.asarray(cap_lo) * 64.0) + k) / 64.0
    tail = np.clip(np.asarray(tail_lo) + u * (np.asarray(tail_hi) - np.asarray(tail_lo)),
                   tail_lo, tail_hi)
    return cap.astype(np.float32), tail.astype(np.float32)


def make_workload(name: str, orders=None, with_samples: bool = True) -> Workload:
    """Build the workload ``name`` (a key of WORKLOADS).  ``orders`` selects a
    subset of its reveal orders (each order has its own seeded stream, so a
    subset is identical to the same rows of the full build)."""
    c = WORKLOADS[name]
    seed = c["seed"]
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    problem = _problem_for(name, rng)
    N = problem.n_cells
    if c.get("structure"):
        cap_lo0, cap_hi0, tail_lo0, tail_hi0, truth_cap, truth_tail = _structured_truth(name, problem, rng)
    else:
        cap_lo0, cap_hi0, tail_lo0, tail_hi0 = _initial_intervals(name, problem, rng)
        truth_cap, truth_tail = _draw_inside(rng, cap_lo0, cap_hi0, tail_lo0, tail_hi0)
    if c["cand"][0] == "subset":
        cand = np.sort(rng.choice(N, size=c["cand"][1], replace=False)).astype(np.int32)
    else:
        cand = np.arange(N, dtype=np.int32)

    all_orders = np.arange(c["orders"])
    sel = all_orders if orders is None else np.asarray(orders, dtype=np.int64)
    O, E, S = len(sel), len(cand), c["samples"]
    cap_lo = np.zeros((O, N), np.float32)
    cap_hi = np.zeros((O, N), np.float32)
    tail_lo = np.zeros((O, N), np.float32)
    tail_hi = np.zeros((O, N), np.float32)
    measured = np.zeros((O, N), np.uint8)
    cap_s = np.zeros((O, E, S), np.float32) if with_samples else None
    tail_s = np.zeros((O, E, S), np.float32) if with_samples else None
    for j, o in enumerate(sel):
        orng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1, int(o)])))
        cl, ch, tl, th = cap_lo0.copy(), cap_hi0.copy(), tail_lo0.copy(), tail_hi0.copy()
        ms = np.zeros(N, np.uint8)
        if c["reveal"]:
            perm = orng.permutation(N)
            k = int(orng.integers(0, N))
            rev = perm[:k]
            cl[rev] = ch[rev] = truth_cap[rev]
            tl[rev] = th[rev] = truth_tail[rev]
            ms[rev] = 1
        cap_lo[j], cap_hi[j], tail_lo[j], tail_hi[j], measured[j] = cl, ch, tl, th, ms
        if with_samples:
            srng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 2, int(o)])))
            cs, ts = _draw_inside(srng, cl[cand], ch[cand], tl[cand], th[cand], shape=(E, S))
            cap_s[j], tail_s[j] = cs, ts
    iv = Intervals(cap_lo, cap_hi, tail_lo, tail_hi, measured)
    return Workload(name, seed, problem, iv, cand, cap_s, tail_s,
                    truth_cap.astype(np.float32), truth_tail.astype(np.float32), sel, S, dict(c))


def seeded_tiles(w: Workload, n: int, seed: int) -> list:
    """n (order, candidate) tiles of a workload whose candidate is unmeasured
    in that order, drawn by a seeded permutation (all of them when n is
    larger); the subsets on which the large workloads are checked and timed
    against the oracle."""
    meas = np.asarray(w.intervals.measured)[:, np.asarray(w.cand)].astype(bool)
    O, E = meas.shape
    live = [(o, e) for o in range(O) for e in range(E) if not meas[o, e]]
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 5])))
    pick = rng.permutation(len(live))[: min(n, len(live))]
    return [live[j] for j in sorted(pick)]


def tile_mask(w: Workload, tiles) -> np.ndarray:
    """[O][E] uint8 mask of the given (order, candidate) tiles."""
    m = np.zeros((np.asarray(w.intervals.measured).shape[0], len(w.cand)), np.uint8)
    for o, e in tiles:
        m[o, e] = 1
    return m


def random_point_tables(problem: Problem, n: int, seed: int, cap_range=(0.0, 4.0),
                        tail_range=(1.0, 60.0)):
    """n dense point realisations (cap[n][N], tail[n][N]) for solve tests:
    capacities on the 1/64 grid (zero allowed), tails uniform."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7])))
    N = problem.n_cells
    cap = np.rint(rng.uniform(*cap_range, size=(n, N)) * 64.0) / 64.0
    tail = rng.uniform(*tail_range, size=(n, N))
    return cap.astype(np.float32), tail.astype(np.float32)


def random_problem(seed: int, K: int, tp, G: int, n_levels: int, critical: bool = False) -> Problem:
    """A small random problem for brute-force comparisons."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 9])))
    levels = np.sort(rng.choice(np.arange(1, 33) * 0.25, size=n_levels, replace=False))
    demand = np.rint(rng.uniform(0.5, 8.0, size=K) * 4.0) / 4.0
    slo = rng.choice(np.array([10.0, 30.0, 60.0]), size=K)
    floor = None
    if critical:
        floor = np.where(rng.random(K) < 0.5, np.rint(rng.uniform(0.25, 4.0, size=K) * 4) / 4, 0.0)
    return Problem(tp=tp, levels=levels, demand=demand, slo=slo, budget=G, floor_rps=floor)


# --------------------------------------------- several metrics per cell --
@dataclass
class PolicyInputs:
    """A second tail metric (TTFT-p99) and a success probability per cell
    for a workload, with the class policy that bounds them (Section 5: chat
    success >= 99%, TTFT-p99 <= 2 s, completion-p99 <= 30 s; code success
    >= 99%, TTFT-p99 <= 5 s).  Metric 0 is the workload's own tail
    (completion), metric 1 the TTFT.  Revealed cells hold the hidden truth."""
    limit: np.ndarray        # [K][2] per-class limits (completion, TTFT)
    success_min: np.ndarray  # [K]
    tail_lo: np.ndarray      # [O][N][2]
    tail_hi: np.ndarray      # [O][N][2]
    succ_lo: np.ndarray      # [O][N]
    succ_hi: np.ndarray      # [O][N]
    truth_tail: np.ndarray   # [N][2]
    truth_succ: np.ndarray   # [N]
    tail_s: np.ndarray       # [O][E][S][2] or None
    succ_s: np.ndarray       # [O][E][S] or None


def make_policy_inputs(w: Workload, with_samples: bool = True) -> PolicyInputs:
    """TTFT intervals (lognormal around a quarter of the class's TTFT limit,
    growing with load, shrinking with TP like the completion tail) and
    success intervals near the 99% floor, drawn with the workload's seed."""
    p = w.problem
    K, T, B, N = p.n_classes, p.n_tp, p.n_levels, p.n_cells
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, 5])))
    if K == 2:
        ttft_limit = np.array([2.0, 5.0], np.float32)
    else:
        ttft_limit = (np.asarray(p.slo, np.float32) / 10.0).astype(np.float32)
    limit = np.stack([np.asarray(p.slo, np.float32), ttft_limit], axis=1)
    success_min = np.full(K, 0.99, np.float32)
    ttft_lo0 = np.zeros(N, np.float32)
    ttft_hi0 = np.zeros(N, np.float32)
    succ_lo0 = np.zeros(N, np.float32)
    succ_hi0 = np.zeros(N, np.float32)
    for i in range(K):
        for t in range(T):
            rho = TAIL_TP_FACTOR[int(p.tp[t])]
            for b in range(B):
                cell = p.cell(i, t, b)
                med = (float(ttft_limit[i]) / 4.0) * (1.0 + float(p.levels[b])) ** 0.5 * rho
                lo = np.float32(med * np.exp(0.4 * rng.standard_normal()))
                ttft_lo0[cell] = lo
                ttft_hi0[cell] = np.float32(float(lo) * (1.0 + rng.uniform(0.1, 0.4)))
                hi = np.float32(1.0 - 10.0 ** (-rng.uniform(2.0, 4.0)))
                succ_hi0[cell] = hi
                succ_lo0[cell] = np.float32(max(0.0, float(hi) - rng.uniform(0.0, 0.005)))
    truth_ttft = np.clip(ttft_lo0 + rng.random(N).astype(np.float32) * (ttft_hi0 - ttft_lo0),
                         ttft_lo0, ttft_hi0).astype(np.float32)
    truth_succ = np.clip(succ_lo0 + rng.random(N).astype(np.float32) * (succ_hi0 - succ_lo0),
                         succ_lo0, succ_hi0).astype(np.float32)
    O = w.n_orders
    m = w.intervals.measured.astype(bool)
    ttft_lo = np.where(m, truth_ttft, ttft_lo0).astype(np.float32)
    ttft_hi = np.where(m, truth_ttft, ttft_hi0).astype(np.float32)
    succ_lo = np.where(m, truth_succ, succ_lo0).astype(np.float32)
    succ_hi = np.where(m, truth_succ, succ_hi0).astype(np.float32)
    tail_lo = np.stack([w.intervals.tail_lo, ttft_lo], axis=-1).astype(np.float32)
    tail_hi = np.stack([w.intervals.tail_hi, ttft_hi], axis=-1).astype(np.float32)
    truth_tail = np.stack([w.truth_tail, truth_ttft], axis=-1).astype(np.float32)
    tail_s = succ_s = None
    if with_samples and w.cap_s is not None:
        E, S = len(w.cand), w.n_samples
        tail_s = np.zeros((O, E, S, 2), np.float32)
        succ_s = np.zeros((O, E, S), np.float32)
        tail_s[..., 0] = w.tail_s
        for j, o in enumerate(w.orders):
            srng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, 6, int(o)])))
            lo, hi = ttft_lo[j][w.cand][:, None], ttft_hi[j][w.cand][:, None]
            tail_s[j, :, :, 1] = np.clip(lo + srng.random((E, S)).astype(np.float32) * (hi - lo), lo, hi)
            lo, hi = succ_lo[j][w.cand][:, None], succ_hi[j][w.cand][:, None]
            succ_s[j] = np.clip(lo + srng.random((E, S)).astype(np.float32) * (hi - lo), lo, hi)
    return PolicyInputs(limit, success_min, tail_lo, tail_hi, succ_lo, succ_hi, truth_tail, truth_succ,
                        tail_s, succ_s)


def interval_realisations(w: Workload, n: int, seed: int = 11):
    """n point realisations of a workload's uncertainty: realisation j draws
    every cell of order j mod O uniformly inside its intervals (capacity on
    the 1/64 req/s grid, tail in binary32).  Returns cap, tail [n][N]."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, seed, 8])))
    iv = w.intervals
    O, N = iv.cap_lo.shape
    rows = np.arange(n) % O
    lo, hi = iv.cap_lo[rows], iv.cap_hi[rows]
    k = np.floor(rng.random((n, N)) * (np.rint((hi - lo) * 64.0) + 1.0))
    cap = (lo + k / 64.0).astype(np.float32)
    tl, th = iv.tail_lo[rows], iv.tail_hi[rows]
    tail = np.clip(tl + rng.random((n, N)).astype(np.float32) * (th - tl), tl, th).astype(np.float32)
    return cap, tail
