"""CPU oracle for FleetSieve -- TEST INFRASTRUCTURE ONLY.

Python access (ctypes) to ``fs_oracle.c``: the plain, slow, binary32-exact
reference implementation of the fleet allocation (Section 3, Eq. 1-5), the
acquisition score (Section 4.3) and the decision certificate (Section 4.2).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path and
imports nothing from it.  A problem is any object with the attributes
``tp, levels, demand, slo, floor_rps, budget`` (numpy arrays / int).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fs_oracle.c")
# FLEETSIEVE_ORACLE_LIB selects another build of fs_oracle.c (for example
# one compiled with sanitizers); the default is the one build() writes here.
_BUILT = os.path.join(_HERE, "liboracle.so")
_LIB = os.environ.get("FLEETSIEVE_ORACLE_LIB") or _BUILT

MAX_CLASSES = 64
UNDECIDED, CERTIFIED_FEASIBLE, CERTIFIED_INFEASIBLE = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc: binary32 arithmetic, no contraction."""
    if force or not os.path.exists(_BUILT):
        tmp = _BUILT + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True, cwd=_HERE)
        os.replace(tmp, _BUILT)
    return _BUILT


class _Problem(ctypes.Structure):
    _fields_ = [("n_classes", ctypes.c_int32), ("n_tp", ctypes.c_int32),
                ("n_levels", ctypes.c_int32), ("budget", ctypes.c_int32),
                ("tp", ctypes.POINTER(ctypes.c_int32)),
                ("levels", ctypes.POINTER(ctypes.c_float)),
                ("demand", ctypes.POINTER(ctypes.c_float)),
                ("slo", ctypes.POINTER(ctypes.c_float)),
                ("floor_rps", ctypes.POINTER(ctypes.c_float))]


class _Alloc(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("floors_met", ctypes.c_int32),
                ("gpus", ctypes.c_int32), ("goodput", ctypes.c_float),
                ("tp_index", ctypes.c_int32 * MAX_CLASSES),
                ("replicas", ctypes.c_int32 * MAX_CLASSES)]


@dataclass
class Alloc:
    tau: float
    floors_met: int
    gpus: int
    goodput: float
    tp_index: list   # -1 = empty
    replicas: list
    goodput64: float = None  # whole objective only: level (3)'s binary64 total

    def tp(self, problem) -> list:
        """GPUs per replica per class (0 = empty)."""
        return [0 if t < 0 else int(problem.tp[t]) for t in self.tp_index]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P, A = ctypes.POINTER(_Problem), ctypes.POINTER(_Alloc)
        fp, u8p, i32p, f64p = (ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_uint8),
                               ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double))
        lib.orc_check_problem.argtypes = [P]
        lib.orc_bucket.argtypes = [P, ctypes.c_int, ctypes.c_int]
        lib.orc_fulfillment.argtypes = [P, ctypes.c_int, ctypes.c_float, ctypes.c_float, ctypes.c_int]
        lib.orc_fulfillment.restype = ctypes.c_float
        for name in ("orc_solve_brute", "orc_solve_dp", "orc_solve_threshold"):
            getattr(lib, name).argtypes = [P, fp, fp, A]
        lib.orc_solve_batch.argtypes = [P, fp, fp, ctypes.c_int64, A, ctypes.c_int]
        lib.orc_score.argtypes = [P, ctypes.c_int32, fp, fp, fp, fp, u8p, i32p, ctypes.c_int32,
                                  fp, fp, ctypes.c_int32, f64p, f64p, i32p, fp, u8p, ctypes.c_int]
        lib.orc_certify.argtypes = [P, ctypes.c_int32, fp, fp, fp, fp, u8p, ctypes.c_float,
                                    i32p, A, A, f64p]
        for name in ("orc_solve_lex", "orc_solve_lex_brute"):
            getattr(lib, name).argtypes = [P, fp, fp, A, f64p]
        lib.orc_certify_lex.argtypes = [P, ctypes.c_int32, fp, fp, fp, fp, u8p, ctypes.c_float,
                                        i32p, A, A, f64p, f64p]
        lib.orc_score_lex.argtypes = [P, ctypes.c_int32, fp, fp, fp, fp, u8p, i32p, ctypes.c_int32,
                                      fp, fp, ctypes.c_int32, f64p, f64p, f64p, f64p, i32p, u8p, ctypes.c_int]
        lib.orc_pairwise_sum.argtypes = [f64p, ctypes.c_int64]
        lib.orc_pairwise_sum.restype = ctypes.c_double
        _lib = lib
    return _lib


def _ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


class _ProblemRef:
    """Holds the numpy buffers alive while the C struct points at them."""

    def __init__(self, problem):
        self.tp = np.ascontiguousarray(problem.tp, dtype=np.int32)
        self.levels = np.ascontiguousarray(problem.levels, dtype=np.float32)
        self.demand = np.ascontiguousarray(problem.demand, dtype=np.float32)
        self.slo = np.ascontiguousarray(problem.slo, dtype=np.float32)
        fl = getattr(problem, "floor_rps", None)
        self.floor = None if fl is None else np.ascontiguousarray(fl, dtype=np.float32)
        self.s = _Problem(len(self.demand), len(self.tp), len(self.levels), int(problem.budget),
                          _ptr(self.tp, ctypes.c_int32), _ptr(self.levels, ctypes.c_float),
                          _ptr(self.demand, ctypes.c_float), _ptr(self.slo, ctypes.c_float),
                          None if self.floor is None else _ptr(self.floor, ctypes.c_float))
        self.n_cells = len(self.demand) * len(self.tp) * len(self.levels)


def _alloc_out(a: _Alloc, k: int) -> Alloc:
    return Alloc(float(np.float32(a.tau)), int(a.floors_met), int(a.gpus), float(np.float32(a.goodput)),
                 [int(a.tp_index[i]) for i in range(k)], [int(a.replicas[i]) for i in range(k)])


def check_problem(problem) -> bool:
    ref = _ProblemRef(problem)
    return _load().orc_check_problem(ctypes.byref(ref.s)) == 0


def bucket(problem, i: int, r: int) -> int:
    ref = _ProblemRef(problem)
    return int(_load().orc_bucket(ctypes.byref(ref.s), i, r))


def fulfillment(problem, i: int, cap: float, tail: float, r: int) -> np.float32:
    ref = _ProblemRef(problem)
    return np.float32(_load().orc_fulfillment(ctypes.byref(ref.s), i, cap, tail, r))


def solve(problem, cap, tail, method: str = "dp") -> Alloc:
    """Solve the allocation on one point realisation (cap[N], tail[N]).
    Methods dp / brute / threshold: objective levels (1)-(2) with the
    fewer-GPUs, smaller-TP tie-breaks; lex / lex_brute: the whole objective,
    levels (1)-(4)."""
    ref = _ProblemRef(problem)
    cap = np.ascontiguousarray(cap, dtype=np.float32)
    tail = np.ascontiguousarray(tail, dtype=np.float32)
    assert cap.shape == (ref.n_cells,) and tail.shape == (ref.n_cells,)
    out = _Alloc()
    if method in ("lex", "lex_brute"):
        gp = ctypes.c_double()
        fn = "orc_solve_lex" if method == "lex" else "orc_solve_lex_brute"
        rc = getattr(_load(), fn)(ctypes.byref(ref.s), _ptr(cap, ctypes.c_float), _ptr(tail, ctypes.c_float),
                                  ctypes.byref(out), ctypes.byref(gp))
        if rc != 0:
            raise ValueError(f"oracle {method} solve failed ({rc})")
        a = _alloc_out(out, len(ref.demand))
        a.goodput64 = float(gp.value)
        return a
    fn = {"dp": "orc_solve_dp", "brute": "orc_solve_brute", "threshold": "orc_solve_threshold"}[method]
    rc = getattr(_load(), fn)(ctypes.byref(ref.s), _ptr(cap, ctypes.c_float), _ptr(tail, ctypes.c_float),
                              ctypes.byref(out))
    if rc != 0:
        raise ValueError(f"oracle {method} solve failed ({rc})")
    return _alloc_out(out, len(ref.demand))


def solve_batch(problem, cap, tail, n_threads: int = 1) -> list:
    ref = _ProblemRef(problem)
    cap = np.ascontiguousarray(cap, dtype=np.float32).reshape(-1, ref.n_cells)
    tail = np.ascontiguousarray(tail, dtype=np.float32).reshape(-1, ref.n_cells)
    n = cap.shape[0]
    out = (_Alloc * max(n, 1))()
    rc = _load().orc_solve_batch(ctypes.byref(ref.s), _ptr(cap, ctypes.c_float), _ptr(tail, ctypes.c_float),
                                 n, out, n_threads)
    if rc != 0:
        raise ValueError("oracle batch solve failed")
    return [_alloc_out(out[j], len(ref.demand)) for j in range(n)]


@dataclass
class ScoreResult:
    score: np.ndarray     # [O][E] float64
    gap_now: np.ndarray   # [O] float64
    best: np.ndarray      # [O] int32
    tau_dump: np.ndarray  # [O][E][S][2] float32 or None


def score(problem, intervals, cand, cap_s, tail_s, tile_mask=None, dump: bool = True,
          n_threads: int = 1) -> ScoreResult:
    """Acquisition scores.  ``intervals`` has cap_lo, cap_hi, tail_lo,
    tail_hi ([O][N] float32) and measured ([O][N] uint8)."""
    ref = _ProblemRef(problem)
    N = ref.n_cells
    cl = np.ascontiguousarray(intervals.cap_lo, dtype=np.float32).reshape(-1, N)
    O = cl.shape[0]
    ch = np.ascontiguousarray(intervals.cap_hi, dtype=np.float32).reshape(O, N)
    tl = np.ascontiguousarray(intervals.tail_lo, dtype=np.float32).reshape(O, N)
    th = np.ascontiguousarray(intervals.tail_hi, dtype=np.float32).reshape(O, N)
    ms = np.ascontiguousarray(intervals.measured, dtype=np.uint8).reshape(O, N)
    cand = np.ascontiguousarray(cand, dtype=np.int32)
    E = len(cand)
    S = max(int(np.shape(cap_s)[-1]), 1)
    cs = np.ascontiguousarray(cap_s, dtype=np.float32)
    ts = np.ascontiguousarray(tail_s, dtype=np.float32)
    if cs.size == 0:
        cs = np.zeros((O, E, S), np.float32)
        ts = np.zeros((O, E, S), np.float32)
    cs, ts = cs.reshape(O, E, S), ts.reshape(O, E, S)
    sc = np.zeros((O, E), dtype=np.float64)
    gap = np.zeros(O, dtype=np.float64)
    best = np.full(O, -1, dtype=np.int32)
    td = np.zeros((O, E, S, 2), dtype=np.float32) if dump else None
    tm = None if tile_mask is None else np.ascontiguousarray(tile_mask, dtype=np.uint8).reshape(O * E)
    rc = _load().orc_score(ctypes.byref(ref.s), O, _ptr(cl, ctypes.c_float), _ptr(ch, ctypes.c_float),
                           _ptr(tl, ctypes.c_float), _ptr(th, ctypes.c_float), _ptr(ms, ctypes.c_uint8),
                           _ptr(cand, ctypes.c_int32), E, _ptr(cs, ctypes.c_float), _ptr(ts, ctypes.c_float),
                           S, _ptr(sc, ctypes.c_double), _ptr(gap, ctypes.c_double),
                           _ptr(best, ctypes.c_int32), None if td is None else _ptr(td, ctypes.c_float),
                           None if tm is None else _ptr(tm, ctypes.c_uint8), n_threads)
    if rc != 0:
        raise ValueError("oracle score failed")
    return ScoreResult(sc, gap, best, td)


@dataclass
class CertifyResult:
    state: np.ndarray   # [O] int32
    gap: np.ndarray     # [O] float64
    cons: list          # [O] Alloc (conservative, A-)
    opt: list           # [O] Alloc (optimistic, A+)


def certify(problem, intervals, eps: float = 0.05) -> CertifyResult:
    ref = _ProblemRef(problem)
    N = ref.n_cells
    cl = np.ascontiguousarray(intervals.cap_lo, dtype=np.float32).reshape(-1, N)
    O = cl.shape[0]
    ch = np.ascontiguousarray(intervals.cap_hi, dtype=np.float32).reshape(O, N)
    tl = np.ascontiguousarray(intervals.tail_lo, dtype=np.float32).reshape(O, N)
    th = np.ascontiguousarray(intervals.tail_hi, dtype=np.float32).reshape(O, N)
    ms = np.ascontiguousarray(intervals.measured, dtype=np.uint8).reshape(O, N)
    state = np.zeros(O, dtype=np.int32)
    gap = np.zeros(O, dtype=np.float64)
    cons = (_Alloc * max(O, 1))()
    opt = (_Alloc * max(O, 1))()
    rc = _load().orc_certify(ctypes.byref(ref.s), O, _ptr(cl, ctypes.c_float), _ptr(ch, ctypes.c_float),
                             _ptr(tl, ctypes.c_float), _ptr(th, ctypes.c_float), _ptr(ms, ctypes.c_uint8),
                             float(eps), _ptr(state, ctypes.c_int32), cons, opt, _ptr(gap, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle certify failed")
    k = len(ref.demand)
    return CertifyResult(state, gap, [_alloc_out(cons[o], k) for o in range(O)],
                         [_alloc_out(opt[o], k) for o in range(O)])


@dataclass
class CertifyLexResult:
    state: np.ndarray   # [O] int32
    gap_mm: np.ndarray  # [O] float64, tau+ - tau-
    gap_gp: np.ndarray  # [O] float64, |gp+ - gp-| / max(gp+, gp-)
    cons: list          # [O] Alloc under the whole objective (A-)
    opt: list           # [O] Alloc (A+)


def certify_lex(problem, intervals, eps: float = 0.05) -> CertifyLexResult:
    """Certificate with the stage-wise gap (Section 4.2) under the whole
    lexicographic objective."""
    ref = _ProblemRef(problem)
    N = ref.n_cells
    cl = np.ascontiguousarray(intervals.cap_lo, dtype=np.float32).reshape(-1, N)
    O = cl.shape[0]
    ch = np.ascontiguousarray(intervals.cap_hi, dtype=np.float32).reshape(O, N)
    tl = np.ascontiguousarray(intervals.tail_lo, dtype=np.float32).reshape(O, N)
    th = np.ascontiguousarray(intervals.tail_hi, dtype=np.float32).reshape(O, N)
    ms = np.ascontiguousarray(intervals.measured, dtype=np.uint8).reshape(O, N)
    state = np.zeros(O, dtype=np.int32)
    gmm = np.zeros(O, dtype=np.float64)
    ggp = np.zeros(O, dtype=np.float64)
    cons = (_Alloc * max(O, 1))()
    opt = (_Alloc * max(O, 1))()
    rc = _load().orc_certify_lex(ctypes.byref(ref.s), O, _ptr(cl, ctypes.c_float), _ptr(ch, ctypes.c_float),
                                 _ptr(tl, ctypes.c_float), _ptr(th, ctypes.c_float), _ptr(ms, ctypes.c_uint8),
                                 float(eps), _ptr(state, ctypes.c_int32), cons, opt, _ptr(gmm, ctypes.c_double),
                                 _ptr(ggp, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle certify failed")
    k = len(ref.demand)
    return CertifyLexResult(state, gmm, ggp, [_alloc_out(cons[o], k) for o in range(O)],
                            [_alloc_out(opt[o], k) for o in range(O)])


@dataclass
class ScoreLexResult:
    score_mm: np.ndarray  # [O][E] expected max-min stage reduction
    score_gp: np.ndarray  # [O][E] expected goodput stage reduction
    gap_mm: np.ndarray    # [O]
    gap_gp: np.ndarray    # [O]
    best: np.ndarray      # [O]


def score_lex(problem, intervals, cand, cap_s, tail_s, tile_mask=None, n_threads: int = 1) -> ScoreLexResult:
    """Acquisition scores with the stage-wise gap under the whole objective
    (orc_score_lex); tiles outside tile_mask are left 0."""
    ref = _ProblemRef(problem)
    N = ref.n_cells
    cl = np.ascontiguousarray(intervals.cap_lo, dtype=np.float32).reshape(-1, N)
    O = cl.shape[0]
    ch = np.ascontiguousarray(intervals.cap_hi, dtype=np.float32).reshape(O, N)
    tl = np.ascontiguousarray(intervals.tail_lo, dtype=np.float32).reshape(O, N)
    th = np.ascontiguousarray(intervals.tail_hi, dtype=np.float32).reshape(O, N)
    ms = np.ascontiguousarray(intervals.measured, dtype=np.uint8).reshape(O, N)
    cand = np.ascontiguousarray(cand, dtype=np.int32)
    E = len(cand)
    cs = np.ascontiguousarray(cap_s, dtype=np.float32).reshape(O, E, -1)
    ts = np.ascontiguousarray(tail_s, dtype=np.float32).reshape(O, E, -1)
    S = cs.shape[2]
    smm = np.zeros((O, E), np.float64)
    sgp = np.zeros((O, E), np.float64)
    gmm = np.zeros(O, np.float64)
    ggp = np.zeros(O, np.float64)
    best = np.zeros(O, np.int32)
    mask = None if tile_mask is None else np.ascontiguousarray(tile_mask, dtype=np.uint8).reshape(O, E)
    rc = _load().orc_score_lex(ctypes.byref(ref.s), O, _ptr(cl, ctypes.c_float), _ptr(ch, ctypes.c_float),
                               _ptr(tl, ctypes.c_float), _ptr(th, ctypes.c_float), _ptr(ms, ctypes.c_uint8),
                               _ptr(cand, ctypes.c_int32), E, _ptr(cs, ctypes.c_float), _ptr(ts, ctypes.c_float), S,
                               _ptr(smm, ctypes.c_double), _ptr(sgp, ctypes.c_double), _ptr(gmm, ctypes.c_double),
                               _ptr(ggp, ctypes.c_double), _ptr(best, ctypes.c_int32),
                               None if mask is None else _ptr(mask, ctypes.c_uint8), int(n_threads))
    if rc != 0:
        raise ValueError("oracle score failed")
    return ScoreLexResult(smm, sgp, gmm, ggp, best)


def pairwise_sum(x) -> float:
    x = np.ascontiguousarray(x, dtype=np.float64)
    return float(_load().orc_pairwise_sum(_ptr(x, ctypes.c_double), len(x)))


# ---------------------------------------------------------- profiling loop --
# Duration of one profiling cell; a reveal costs this times the cell's TP
# degree in GPU-seconds (Section 5: 300-second cells, cost = duration x GPUs).
CELL_SECONDS = 300.0
POLICY_SCORE, POLICY_ORDER = 0, 1


@dataclass
class LoopResult:
    state: np.ndarray        # [O] int32 certificate state when the loop ended
    finished: np.ndarray     # [O] uint8: 1 = certified, or no unmeasured candidate was left
    rounds: np.ndarray       # [O] int32 reveals made
    gpu_seconds: np.ndarray  # [O] float64: CELL_SECONDS x TP summed over the reveals
    reveals: np.ndarray      # [O][max_rounds] int32 candidate revealed in each round, -1 after the end
    final: list              # [O] Alloc returned: A- when certified, else the best measured allocation
    tau_truth: np.ndarray    # [O] float32: the returned allocation's objective on the true table
    tau_oracle: np.ndarray   # [O] float32: the optimum of the true table
    regret: np.ndarray       # [O] float64: tau_oracle - tau_truth


def value_on_table(problem, alloc: Alloc, cap, tail) -> np.float32:
    """Objective level (2) of a fixed allocation on a point table: the
    smallest fulfillment over the classes, an empty class counting 0."""
    ref = _ProblemRef(problem)
    K, T, B = len(ref.demand), len(ref.tp), len(ref.levels)
    v = np.float32(np.inf)
    for i in range(K):
        r = alloc.replicas[i]
        if r == 0:
            return np.float32(0.0)
        b = bucket(problem, i, r)
        cell = (i * T + alloc.tp_index[i]) * B + b
        v = min(v, fulfillment(problem, i, float(cap[cell]), float(tail[cell]), r))
    return np.float32(v)


def profile_loop(problem, intervals, truth_cap, truth_tail, cand, cap_s, tail_s, eps: float = 0.05,
                 policy: int = POLICY_SCORE, order=None, max_rounds: int = None,
                 n_threads: int = 1, objective: str = "maxmin", refit: bool = False) -> LoopResult:
    """Algorithm 1 (the profiling loop) for O independent trajectories, each
    starting from its own row of ``intervals`` (the common initial design).
    Per round, for every trajectory still running: the conservative and
    optimistic allocations and the certificate (Section 4.2); a certified
    state (feasible or infeasible) ends the trajectory and returns A-;
    otherwise one unmeasured candidate is revealed -- its cell's intervals
    collapse to the true values truth_cap[o][cell], truth_tail[o][cell] and
    it becomes measured -- at a cost of CELL_SECONDS x TP GPU-seconds.  The
    revealed candidate is the score's argmax (Section 4.3; POLICY_SCORE) or,
    for the comparison, the first unmeasured one in order[o] (POLICY_ORDER,
    e.g. a uniform random permutation).  A trajectory with no unmeasured
    candidate left ends undecided (the certificate of its final intervals is
    evaluated first, so a last reveal can still certify) and returns the best
    measured feasible allocation (Algorithm 1's last line): the optimum of its
    table with every unmeasured cell infeasible (tail +inf) and every measured
    cell at its measured values; so does a trajectory stopped by the round
    limit.  With
    objective="lex" the certificate and the score are the stage-wise ones
    under the whole objective (certify_lex, score_lex) and A- is that
    objective's allocation.  With
    refit=True every round starts with refit_intervals (Algorithm 1's fit
    step) of the trajectory's initial intervals with its revealed cells, the
    certificate and score use the refitted intervals, and the score's
    samples are clamped into them.  The
    allocation's value on the true table gives the decision regret against
    the true optimum.  The intervals are not refitted
    between rounds; the samples of a candidate stay valid because its
    intervals only change when it is revealed.  After max_rounds reveals
    (default: the number of candidates) the trajectory stops undecided."""
    ref = _ProblemRef(problem)
    N = ref.n_cells
    cl = np.array(intervals.cap_lo, dtype=np.float32).reshape(-1, N)
    O = cl.shape[0]
    ch = np.array(intervals.cap_hi, dtype=np.float32).reshape(O, N)
    tl = np.array(intervals.tail_lo, dtype=np.float32).reshape(O, N)
    th = np.array(intervals.tail_hi, dtype=np.float32).reshape(O, N)
    ms = np.array(intervals.measured, dtype=np.uint8).reshape(O, N)
    tc = np.asarray(truth_cap, dtype=np.float32).reshape(O, N)
    tt = np.asarray(truth_tail, dtype=np.float32).reshape(O, N)
    cand = np.asarray(cand, dtype=np.int32)
    E = len(cand)
    R = E if max_rounds is None else int(max_rounds)
    state = np.zeros(O, np.int32)
    finished = np.zeros(O, np.uint8)
    rounds = np.zeros(O, np.int32)
    gpu_s = np.zeros(O, np.float64)
    reveals = np.full((O, R), -1, np.int32)
    final = [None] * O
    running = np.ones(O, bool)

    class _Rows:  # the running trajectories' intervals, for the primitives
        def __init__(self, idx):
            self.cap_lo, self.cap_hi, self.tail_lo, self.tail_hi = cl[idx], ch[idx], tl[idx], th[idx]
            self.measured = ms[idx]

    for rnd in range(R + 1):
        idx = np.nonzero(running)[0]
        if len(idx) == 0:
            break
        # the refit is a function of the initial intervals and the revealed
        # cells, recomputed every round (the trajectory's own arrays keep the
        # unrefitted intervals)
        rows = refit_intervals(problem, _Rows(idx)) if refit else _Rows(idx)
        cert = certify(problem, rows, eps) if objective == "maxmin" else certify_lex(problem, rows, eps)
        for j, o in enumerate(idx):
            state[o] = cert.state[j]
            final[o] = cert.cons[j]
            if cert.state[j] != UNDECIDED:
                finished[o] = 1
                running[o] = False
            elif all(ms[o, c] for c in cand):  # no unmeasured candidate: A- undecided
                finished[o] = 1
                running[o] = False
        if rnd == R:
            break
        idx = np.nonzero(running)[0]
        if len(idx) == 0:
            break
        if policy == POLICY_SCORE:
            cs, ts = np.asarray(cap_s)[idx], np.asarray(tail_s)[idx]
            rows = _Rows(idx)
            if refit:
                rows = refit_intervals(problem, rows)
                cs, ts = clamp_samples(rows, cand, cs, ts)
            if objective == "maxmin":
                sc = score(problem, rows, cand, cs, ts, dump=False, n_threads=n_threads)
            else:
                sc = score_lex(problem, rows, cand, cs, ts, n_threads=n_threads)
            picks = [int(b) for b in sc.best]
        else:
            picks = []
            for o in idx:
                pick = -1
                for e in order[o]:
                    if not ms[o, cand[e]]:
                        pick = int(e)
                        break
                picks.append(pick)
        for o, e in zip(idx, picks):
            cell = int(cand[e])
            cl[o, cell] = ch[o, cell] = tc[o, cell]
            tl[o, cell] = th[o, cell] = tt[o, cell]
            ms[o, cell] = 1
            t = int(ref.tp[(cell // len(ref.levels)) % len(ref.tp)])
            gpu_s[o] += CELL_SECONDS * t
            reveals[o, rounds[o]] = e
            rounds[o] += 1

    # A trajectory that ends without a certificate (no unmeasured candidate
    # left, or the round limit) returns Algorithm 1's "best measured feasible
    # allocation": the optimum of the table in which every unmeasured cell is
    # infeasible and every measured cell takes its measured values.
    for o in range(O):
        if state[o] == UNDECIDED:
            masked_tail = np.where(ms[o] != 0, th[o], np.float32(np.inf)).astype(np.float32)
            final[o] = solve(problem, cl[o], masked_tail, "dp" if objective == "maxmin" else "lex")
    tau_truth = np.zeros(O, np.float32)
    tau_oracle = np.zeros(O, np.float32)
    for o in range(O):
        tau_oracle[o] = np.float32(solve(problem, tc[o], tt[o]).tau)
        tau_truth[o] = value_on_table(problem, final[o], tc[o], tt[o])
    regret = tau_oracle.astype(np.float64) - tau_truth.astype(np.float64)
    return LoopResult(state, finished, rounds, gpu_s, reveals, final, tau_truth, tau_oracle, regret)


# ------------------------------------------------------- interval refit --
def _round_down_f32(x: float) -> np.float32:
    """The largest binary32 value not above the binary64 value x."""
    v = np.float32(x)
    if float(v) > x:
        v = np.nextafter(v, np.float32(-np.inf))
    return np.float32(v)


def refit_intervals(problem, intervals):
    """Interval refit of Algorithm 1's fit step under a structural prior
    (Section 4.1: an interior-knee prior combined with the measured cells).
    The prior, as read here: for every class and load level, the capacity
    per GPU (c / t) is unimodal over the TP degrees in ascending order (it
    rises to the knee and falls after it), and for every class and TP degree
    the tail is nondecreasing in the load level.  Consequences drawn from the
    measured cells (their point values), for every unmeasured cell:
      capacity: for measured TP degrees t_a < t < t_b at the same class and
        level, c(t) / t >= min(c(t_a) / t_a, c(t_b) / t_b), so
        cap_lo >= t * min(...) (binary64, rounded down to binary32);
      tail: tail_lo >= the largest measured tail at a lower level of the same
        class and TP, tail_hi <= the smallest measured tail at a higher level.
    A bound that would empty the interval contradicts the prior; that
    quantity keeps its interval.  Measured cells are unchanged.  Returns new
    [O][N] arrays (cap_lo, cap_hi, tail_lo, tail_hi, measured)."""
    from types import SimpleNamespace
    ref = _ProblemRef(problem)
    K, T, B = len(ref.demand), len(ref.tp), len(ref.levels)
    N = K * T * B
    cl = np.array(intervals.cap_lo, dtype=np.float32).reshape(-1, N)
    O = cl.shape[0]
    ch = np.array(intervals.cap_hi, dtype=np.float32).reshape(O, N)
    tl = np.array(intervals.tail_lo, dtype=np.float32).reshape(O, N)
    th = np.array(intervals.tail_hi, dtype=np.float32).reshape(O, N)
    ms = np.array(intervals.measured, dtype=np.uint8).reshape(O, N)
    out_cl, out_tl, out_th = cl.copy(), tl.copy(), th.copy()
    cell = lambda i, t, b: (i * T + t) * B + b
    for o in range(O):
        for i in range(K):
            for b in range(B):
                for t in range(T):
                    c = cell(i, t, b)
                    if ms[o, c]:
                        continue
                    lo = cl[o, c]
                    for a in range(t):
                        for z in range(t + 1, T):
                            ca, cz = cell(i, a, b), cell(i, z, b)
                            if not (ms[o, ca] and ms[o, cz]):
                                continue
                            per_gpu = min(float(cl[o, ca]) / float(ref.tp[a]), float(cl[o, cz]) / float(ref.tp[z]))
                            lo = max(lo, _round_down_f32(float(ref.tp[t]) * per_gpu))
                    if lo <= ch[o, c]:
                        out_cl[o, c] = lo
            for t in range(T):
                for b in range(B):
                    c = cell(i, t, b)
                    if ms[o, c]:
                        continue
                    lo, hi = tl[o, c], th[o, c]
                    for b2 in range(B):
                        c2 = cell(i, t, b2)
                        if not ms[o, c2]:
                            continue
                        if b2 < b:
                            lo = max(lo, tl[o, c2])
                        elif b2 > b:
                            hi = min(hi, tl[o, c2])
                    if lo <= hi:
                        out_tl[o, c], out_th[o, c] = lo, hi
    return SimpleNamespace(cap_lo=out_cl, cap_hi=ch.copy(), tail_lo=out_tl, tail_hi=out_th, measured=ms.copy())


def clamp_samples(intervals, cand, cap_s, tail_s):
    """Samples of each candidate moved into its current intervals
    (min(max(x, lo), hi)); used after a refit."""
    cl = np.asarray(intervals.cap_lo, np.float32)
    O = cl.shape[0]
    cand = np.asarray(cand, np.int64)
    lo_c, hi_c = cl[:, cand][:, :, None], np.asarray(intervals.cap_hi, np.float32)[:, cand][:, :, None]
    lo_t = np.asarray(intervals.tail_lo, np.float32)[:, cand][:, :, None]
    hi_t = np.asarray(intervals.tail_hi, np.float32)[:, cand][:, :, None]
    cs = np.minimum(np.maximum(np.asarray(cap_s, np.float32).reshape(O, len(cand), -1), lo_c), hi_c)
    ts = np.minimum(np.maximum(np.asarray(tail_s, np.float32).reshape(O, len(cand), -1), lo_t), hi_t)
    return cs.astype(np.float32), ts.astype(np.float32)


# ------------------------------------------------ multi-metric feasibility --
@dataclass
class Policy:
    """Class policy of Eq. 5 in full: a configuration is feasible only if
    every tail metric m is within limit[i][m] and (when given) its success
    probability is at least success_min[i].  limit [K][M] (+inf = no limit),
    success_min [K] or None."""
    limit: np.ndarray
    success_min: np.ndarray = None

    @property
    def n_metrics(self) -> int:
        return int(np.asarray(self.limit).shape[1])


def feasible_cells(problem, policy: Policy, tails, success=None) -> np.ndarray:
    """Feasibility of each cell under the class policy (Eq. 5): tails is
    [..., N, M] (metric fastest), success [..., N] or None.  Binary32
    comparisons, inclusive limits."""
    ref = _ProblemRef(problem)
    K, T, B = len(ref.demand), len(ref.tp), len(ref.levels)
    lim = np.asarray(policy.limit, np.float32).reshape(K, -1)
    cls = np.repeat(np.arange(K), T * B)
    tails = np.asarray(tails, np.float32)
    ok = np.all(tails <= lim[cls], axis=-1)
    if policy.success_min is not None:
        smin = np.asarray(policy.success_min, np.float32)
        ok &= np.asarray(success, np.float32) >= smin[cls]
    return ok


def pseudo_tail(ok) -> np.ndarray:
    """A single tail value per cell that carries the policy: 0 when the cell
    is feasible, +inf when it is not; a problem with every SLO at 0 then
    tests exactly the policy."""
    return np.where(ok, np.float32(0.0), np.float32(np.inf)).astype(np.float32)


def feasible_samples(problem, policy: Policy, cand, tail_s, succ_s=None) -> np.ndarray:
    """Feasibility of candidate samples, each judged by its candidate cell's
    class (Eq. 5): tail_s [O][E][S][M], succ_s [O][E][S] or None.  A
    candidate outside the cell range is infeasible."""
    ref = _ProblemRef(problem)
    K, T, B = len(ref.demand), len(ref.tp), len(ref.levels)
    N = K * T * B
    lim = np.asarray(policy.limit, np.float32).reshape(K, -1)
    tail_s = np.asarray(tail_s, np.float32)
    O, E, S, M = tail_s.shape
    out = np.zeros((O, E, S), bool)
    for e, c in enumerate(np.asarray(cand, np.int64)):
        if c < 0 or c >= N:
            continue
        i = int(c) // (T * B)
        ok = np.all(tail_s[:, e] <= lim[i], axis=-1)
        if policy.success_min is not None:
            ok &= np.asarray(succ_s, np.float32)[:, e] >= np.float32(policy.success_min[i])
        out[:, e] = ok
    return out


def reduce_intervals(problem, policy: Policy, intervals, tail_lo_m, tail_hi_m, succ_lo=None, succ_hi=None):
    """Single-metric intervals equivalent to multi-metric ones: the
    conservative side (upper tail bounds, lower success bound) becomes
    tail_hi, the optimistic side (lower tails, upper success) tail_lo."""
    from types import SimpleNamespace
    hi = pseudo_tail(feasible_cells(problem, policy, tail_hi_m, succ_lo))
    lo = pseudo_tail(feasible_cells(problem, policy, tail_lo_m, succ_hi))
    return SimpleNamespace(cap_lo=intervals.cap_lo, cap_hi=intervals.cap_hi, tail_lo=lo, tail_hi=hi,
                           measured=intervals.measured)


def solve_policy_brute(problem, policy: Policy, cap, tails, success=None) -> float:
    """Max-min fulfillment with the full policy applied option by option,
    by enumeration (tiny problems only; objective level (2) without floors):
    each class takes one option (TP t, r replicas) on cell (i, t, bucket(r))
    or nothing, Sum t r <= G."""
    import itertools
    ref = _ProblemRef(problem)
    K, T, B, G = len(ref.demand), len(ref.tp), len(ref.levels), int(problem.budget)
    lim = np.asarray(policy.limit, np.float32).reshape(K, -1)
    tails = np.asarray(tails, np.float32).reshape(K * T * B, -1)
    opts = []
    for i in range(K):
        o = [(0, np.float32(0.0))]
        for t in range(T):
            for r in range(1, G // int(ref.tp[t]) + 1):
                b = bucket(problem, i, r)
                if b < 0:
                    continue
                cell = (i * T + t) * B + b
                ok = bool(np.all(tails[cell] <= lim[i]))
                if policy.success_min is not None:
                    ok = ok and np.float32(success[cell]) >= np.float32(policy.success_min[i])
                cap_r = np.float32(np.float32(r) * np.float32(cap[cell]))
                f = min(np.float32(1.0), np.float32(cap_r / np.float32(ref.demand[i]))) if ok else np.float32(0.0)
                o.append((int(ref.tp[t]) * r, np.float32(f)))
        opts.append(o)
    best = np.float32(0.0)
    for combo in itertools.product(*opts):
        if sum(c for c, _ in combo) <= G:
            best = max(best, min(f for _, f in combo))
    return float(best)
