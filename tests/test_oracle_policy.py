"""Pins of multi-metric feasibility (Eq. 5 with several tail metrics and a
success floor): hand-derived cases under the paper's chat and code policies
(tests/golden/policy_feasibility.json), and brute force with the full policy
applied option by option against the DP on the pseudo-tail reduction (0 when
a cell passes its class's policy, +inf otherwise, every SLO at 0)."""
from types import SimpleNamespace

import numpy as np
import pytest

import oracle
from conftest import load_golden
from paper_2608_19659_amd.synth import Problem, random_point_tables, random_problem


def _zero_slo(p):
    return SimpleNamespace(tp=p.tp, levels=p.levels, demand=p.demand, slo=np.zeros(len(p.demand), np.float32),
                           floor_rps=getattr(p, "floor_rps", None), budget=p.budget)


@pytest.mark.parametrize("case", range(len(load_golden("policy_feasibility.json")["cases"])))
def test_paper_policy_cases(case):
    g = load_golden("policy_feasibility.json")
    c = g["cases"][case]
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=[0.0, 0.0], budget=g["budget"])
    if c.get("capacity_only"):
        pol = oracle.Policy(limit=np.full((2, 2), np.inf, np.float32))
    else:
        pol = oracle.Policy(limit=np.array(g["limit"], np.float32), success_min=np.array(g["success_min"], np.float32))
    ok = oracle.feasible_cells(p, pol, c["tails"], c["success"])
    assert list(ok) == c["feasible"], c["what"]
    a = oracle.solve(_zero_slo(p), np.array(g["cap"], np.float32), oracle.pseudo_tail(ok))
    assert a.tau == np.float32(c["tau"])
    assert [255 if t < 0 else t for t in a.tp_index] == c["tp_index"] and a.replicas == c["replicas"]
    assert oracle.solve_policy_brute(p, pol, g["cap"], c["tails"], c["success"]) == np.float32(c["tau"])


@pytest.mark.parametrize("seed", range(40))
def test_reduction_matches_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    p = random_problem(seed, K=2, tp=[1, 2, 4], G=7, n_levels=3)
    N, M = 18, 3
    cap, _ = random_point_tables(p, 1, seed)
    tails = rng.uniform(0.5, 60.0, size=(N, M)).astype(np.float32)
    succ = rng.uniform(0.97, 1.0, size=N).astype(np.float32)
    lim = rng.choice(np.array([2.0, 5.0, 30.0, np.inf], np.float32), size=(2, M))
    pol = oracle.Policy(limit=lim, success_min=np.array([0.99, 0.98], np.float32) if seed % 2 else None)
    ok = oracle.feasible_cells(p, pol, tails, succ)
    a = oracle.solve(_zero_slo(p), cap[0], oracle.pseudo_tail(ok)).tau
    assert np.float32(a) == np.float32(oracle.solve_policy_brute(p, pol, cap[0], tails, succ))


def test_single_metric_policy_is_the_slo_test():
    """With one metric whose limit is the SLO and no success floor, the
    reduction reproduces the plain tail test of every other call."""
    rng = np.random.default_rng(7)
    p = random_problem(3, K=2, tp=[1, 2, 4, 8], G=16, n_levels=3)
    cap, tail = random_point_tables(p, 4, 3)
    pol = oracle.Policy(limit=np.asarray(p.slo, np.float32)[:, None])
    for j in range(4):
        ok = oracle.feasible_cells(p, pol, tail[j][:, None])
        a = oracle.solve(p, cap[j], tail[j])
        b = oracle.solve(_zero_slo(p), cap[j], oracle.pseudo_tail(ok))
        assert a.tau == b.tau and a.tp_index == b.tp_index and a.replicas == b.replicas


def test_sample_feasibility_is_cell_feasibility_at_the_candidate():
    """A sample of candidate c is judged exactly as cell c would be with the
    sample's metrics in its place; limits are inclusive, NaN fails, and a
    candidate outside the cell range is infeasible."""
    rng = np.random.default_rng(21)
    p = random_problem(5, K=3, tp=[1, 2, 4], G=12, n_levels=2)
    N, M, O, S = p.n_cells, 2, 2, 5
    lim = np.array([[3.0, 1.0], [np.inf, 2.0], [5.0, np.inf]], np.float32)
    pol = oracle.Policy(limit=lim, success_min=np.array([0.99, 0.95, 0.9], np.float32))
    cand = np.array([0, 7, N - 1, 12, N, -1], np.int32)
    tail_s = rng.uniform(0.0, 6.0, size=(O, len(cand), S, M)).astype(np.float32)
    succ_s = rng.uniform(0.85, 1.0, size=(O, len(cand), S)).astype(np.float32)
    tail_s[0, 0, 0] = lim[0]           # exactly at the limits: feasible if success passes
    succ_s[0, 0, 0] = np.float32(0.99)
    tail_s[0, 1, 1, 1] = np.nan
    got = oracle.feasible_samples(p, pol, cand, tail_s, succ_s)
    assert got[0, 0, 0] and not got[0, 1, 1]
    assert not got[:, 4:].any()
    for o in range(O):
        for e, c in enumerate(cand[:4]):
            for s in range(S):
                tails = np.zeros((N, M), np.float32)
                succ = np.ones(N, np.float32)
                tails[c], succ[c] = tail_s[o, e, s], succ_s[o, e, s]
                assert got[o, e, s] == oracle.feasible_cells(p, pol, tails, succ)[c]


def test_interval_sides_hand_derived():
    """The conservative side pairs the upper tail bounds with the LOWER
    success bound, the optimistic side the lower tails with the upper
    success bound (tests/golden/policy_intervals.json): a swapped pairing
    flips cells 1 and 2."""
    g = load_golden("policy_intervals.json")
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"])
    pol = oracle.Policy(limit=np.array(g["limit"], np.float32), success_min=np.array(g["success_min"], np.float32))
    N = p.n_cells
    iv = SimpleNamespace(cap_lo=np.ones((1, N), np.float32), cap_hi=np.ones((1, N), np.float32),
                         tail_lo=np.zeros((1, N), np.float32), tail_hi=np.zeros((1, N), np.float32),
                         measured=np.zeros((1, N), np.uint8))
    a = lambda k: np.array([g[k]], np.float32)
    r = oracle.reduce_intervals(p, pol, iv, a("tail_lo"), a("tail_hi"), a("succ_lo"), a("succ_hi"))
    assert r.tail_hi.tolist() == [g["conservative_tail_hi"]]
    assert r.tail_lo.tolist() == [g["optimistic_tail_lo"]]
    swapped = oracle.reduce_intervals(p, pol, iv, a("tail_lo"), a("tail_hi"), a("succ_hi"), a("succ_lo"))
    assert swapped.tail_hi.tolist() != [g["conservative_tail_hi"]]
    assert swapped.tail_lo.tolist() != [g["optimistic_tail_lo"]]
