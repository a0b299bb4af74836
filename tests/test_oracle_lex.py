"""Pins of the whole lexicographic objective (Section 3: floors, max-min
fulfillment, served goodput, fragmentation) and of the stage-wise
certificate (Section 4.2, Fig. 4a): hand-derived cases on the HW1 instance
(tests/golden/lex_objective.json), brute force over every allocation
against the knapsack, and relations to the max-min solver."""
from types import SimpleNamespace

import numpy as np
import pytest

import oracle
from conftest import load_golden
from paper_2608_19659_amd.synth import Problem, random_point_tables, random_problem

STATES = {"UNDECIDED": 0, "CERTIFIED_FEASIBLE": 1, "CERTIFIED_INFEASIBLE": 2}


def hw1_tables(g, budget, floor=None, code_tail=None, overrides=()):
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=budget,
                floor_rps=None if floor is None else np.array(floor, np.float32))
    cap = np.zeros(p.n_cells, np.float32)
    tail = np.full(p.n_cells, g["tail"], np.float32)
    for i, name in enumerate(("chat", "code")):
        for t in range(p.n_tp):
            for b in range(p.n_levels):
                cap[p.cell(i, t, b)] = g["cap"][name][t]
                if i == 1 and code_tail is not None:
                    tail[p.cell(i, t, b)] = code_tail
    for i, t, b, v in overrides:
        tail[p.cell(i, t, b)] = v
    return p, cap, tail


@pytest.mark.parametrize("case", range(len(load_golden("lex_objective.json")["solves"])))
@pytest.mark.parametrize("method", ["lex", "lex_brute"])
def test_hand_derived_solves(case, method):
    g = load_golden("lex_objective.json")
    c = g["solves"][case]
    p, cap, tail = hw1_tables(g, c["budget"], c.get("floor"), c.get("code_tail"), c.get("tail_override", ()))
    a = oracle.solve(p, cap, tail, method)
    assert a.tau == np.float32(c["tau"]), c["what"]
    assert a.tp(p) == c["tp"] and a.replicas == c["replicas"], (c["what"], a.tp(p), a.replicas)
    assert a.gpus == c["gpus"] and a.goodput64 == c["goodput"] and a.goodput == np.float32(c["goodput"])
    if "maxmin_tp" in c:  # where the max-min tie-breaks decide otherwise
        m = oracle.solve(p, cap, tail, "dp")
        assert m.tp(p) == c["maxmin_tp"] and m.replicas == c["maxmin_replicas"]


@pytest.mark.parametrize("case", range(len(load_golden("lex_objective.json")["certificates"])))
def test_hand_derived_certificates(case):
    g = load_golden("lex_objective.json")
    c = g["certificates"][case]
    p, cap, tail = hw1_tables(g, c["budget"])
    lo = cap.copy()
    lo[c["cell"]] = c["cap_lo"]
    hi = cap.copy()
    if c["measured_cell"]:
        hi[c["cell"]] = c["cap_lo"]
    meas = np.ones(p.n_cells, np.uint8)
    meas[c["cell"]] = c["measured_cell"]
    iv = SimpleNamespace(cap_lo=lo[None], cap_hi=hi[None], tail_lo=tail[None], tail_hi=tail[None],
                         measured=meas[None])
    r = oracle.certify_lex(p, iv, c["eps"])
    assert r.state[0] == STATES[c["state"]], c["what"]
    assert r.gap_mm[0] == c["gap_mm"]
    assert r.gap_gp[0] == c["gap_gp_num"] / c["gap_gp_den"]
    assert r.cons[0].tp(p) == c["cons_tp"] and r.cons[0].replicas == c["cons_replicas"]
    assert r.opt[0].tp(p) == c["opt_tp"] and r.opt[0].replicas == c["opt_replicas"]
    assert oracle.certify(p, iv, c["eps"]).state[0] == STATES[c["maxmin_state"]]


def _random_instance(seed, floors):
    p = random_problem(seed, K=2 + seed % 2, tp=[1, 2, 4], G=6 + seed % 4, n_levels=2, critical=floors)
    cap, tail = random_point_tables(p, 1, seed)
    return p, cap[0], tail[0]


@pytest.mark.parametrize("floors", [False, True])
def test_knapsack_equals_brute_force(floors):
    """Every key of the whole objective, on 150 random tiny instances each."""
    for seed in range(150):
        p, cap, tail = _random_instance(seed, floors)
        a = oracle.solve(p, cap, tail, "lex")
        b = oracle.solve(p, cap, tail, "lex_brute")
        assert (a.tau, a.floors_met, a.gpus) == (b.tau, b.floors_met, b.gpus), seed
        assert a.tp_index == b.tp_index and a.replicas == b.replicas, seed
        assert a.goodput64 == b.goodput64 and np.float32(a.goodput) == np.float32(b.goodput), seed


def _goodput64(p, cap, tail, a):
    """Level (3)'s total of an allocation: served (0 past the SLO) summed in
    binary64 from the last class to the first."""
    total = 0.0
    for i in reversed(range(p.n_classes)):
        if a.replicas[i] == 0:
            continue
        r = a.replicas[i]
        cell = p.cell(i, a.tp_index[i], oracle.bucket(p, i, r))
        if tail[cell] <= p.slo[i]:
            total = float(min(np.float32(p.demand[i]), np.float32(np.float32(r) * cap[cell]))) + total
    return total


@pytest.mark.parametrize("floors", [False, True])
def test_levels_one_and_two_are_kept(floors):
    """The whole objective keeps the max-min solver's tau* and floor outcome,
    serves at least as much as the max-min allocation, and uses at most as
    many GPUs whenever it serves exactly as much."""
    for seed in range(150, 300):
        p, cap, tail = _random_instance(seed, floors)
        a = oracle.solve(p, cap, tail, "lex")
        m = oracle.solve(p, cap, tail, "dp")
        assert a.tau == m.tau and a.floors_met == m.floors_met, seed
        assert a.goodput64 == _goodput64(p, cap, tail, a), seed
        gm = _goodput64(p, cap, tail, m)
        assert a.goodput64 >= gm, seed
        if a.goodput64 == gm:
            assert a.gpus <= m.gpus, seed


def test_certificate_stages():
    """Point intervals close both stages; the max-min stage equals the plain
    certificate's gap; the goodput stage lies in [0, 1]."""
    p = random_problem(8, K=3, tp=[1, 2, 4, 8], G=8, n_levels=3)
    cap, tail = random_point_tables(p, 6, 8)
    rng = np.random.default_rng(8)
    w = rng.uniform(0.0, 0.6, size=cap.shape).astype(np.float32)
    iv = SimpleNamespace(cap_lo=cap, cap_hi=(cap * (1 + w)).astype(np.float32),
                         tail_lo=(tail * (1 - w / 2)).astype(np.float32),
                         tail_hi=(tail * (1 + w)).astype(np.float32), measured=np.zeros(cap.shape, np.uint8))
    r = oracle.certify_lex(p, iv, 0.05)
    m = oracle.certify(p, iv, 0.05)
    np.testing.assert_array_equal(r.gap_mm, m.gap)
    assert ((r.gap_gp >= 0) & (r.gap_gp <= 1)).all() and (r.gap_gp > 0).any()
    pt = SimpleNamespace(cap_lo=cap, cap_hi=cap, tail_lo=tail, tail_hi=tail, measured=np.ones(cap.shape, np.uint8))
    r = oracle.certify_lex(p, pt, 0.0)
    assert (r.gap_mm == 0).all() and (r.gap_gp == 0).all() and (r.state == 1).all()


def _loop_inputs(g, c):
    p, cap, tail = hw1_tables(g, c["budget"])
    cell = c["cand"][0]
    lo, hi, truth = cap.copy(), cap.copy(), cap.copy()
    lo[cell] = min(c["cap_s"])
    hi[cell] = max(c["cap_s"])
    truth[cell] = c["truth_cap"]
    meas = np.ones(p.n_cells, np.uint8)
    meas[cell] = 0
    iv = SimpleNamespace(cap_lo=lo[None], cap_hi=hi[None], tail_lo=tail[None], tail_hi=tail[None],
                         measured=meas[None])
    cs = np.array([[c["cap_s"]]], np.float32)
    ts = np.full_like(cs, g["tail"])
    return p, iv, truth[None], tail[None], np.array(c["cand"], np.int32), cs, ts


@pytest.mark.parametrize("objective", ["lex", "maxmin"])
def test_hand_derived_loop(objective):
    g = load_golden("lex_objective.json")
    c = g["loop"]
    p, iv, tc, tt, cand, cs, ts = _loop_inputs(g, c)
    r = oracle.profile_loop(p, iv, tc, tt, cand, cs, ts, eps=c["eps"], objective=objective)
    want = c[objective]
    assert r.state[0] == STATES[want["state"]] and r.rounds[0] == want["rounds"]
    assert list(r.reveals[0][: want["rounds"]]) == want["reveals"] and r.gpu_seconds[0] == want["gpu_seconds"]
    assert r.final[0].tp(p) == want["final_tp"] and r.final[0].replicas == want["final_replicas"]
    assert r.tau_truth[0] == np.float32(want["tau_truth"]) and r.regret[0] == 0.0


def _score_inputs(g, c):
    p, cap, tail = hw1_tables(g, c["budget"])
    lo, hi = cap.copy(), cap.copy()
    meas = np.ones(p.n_cells, np.uint8)
    for k, v in c["cap_lo"].items():
        lo[int(k)] = v
        meas[int(k)] = 0
    for k, v in c["cap_hi"].items():
        hi[int(k)] = v
    iv = SimpleNamespace(cap_lo=lo[None], cap_hi=hi[None], tail_lo=tail[None], tail_hi=tail[None],
                         measured=meas[None])
    cs = np.array([c["cap_s"]], np.float32)
    return p, iv, np.array(c["cand"], np.int32), cs, np.full_like(cs, g["tail"])


def test_hand_derived_stagewise_score():
    g = load_golden("lex_objective.json")
    c = g["score"]
    p, iv, cand, cs, ts = _score_inputs(g, c)
    r = oracle.score_lex(p, iv, cand, cs, ts)
    assert list(r.score_mm[0]) == c["score_mm"]
    assert list(r.score_gp[0]) == [x / c["score_gp_den"] for x in c["score_gp_num"]]
    assert r.gap_gp[0] == c["gap_gp_num"] / c["score_gp_den"] and r.best[0] == c["best"]
    assert oracle.score(p, iv, cand, cs, ts).best[0] == c["maxmin_best"]


@pytest.mark.parametrize("name,orders", [("paper-shaped-2class-G16", [0, 3, 5]), ("4class-G64", [1])])
def test_stagewise_score_keeps_the_maxmin_stage(name, orders):
    """The max-min stage of the stage-wise score is the plain score, bit for
    bit (tau* is the same under both objectives), and measured candidates
    score (0, 0) and are never picked."""
    from paper_2608_19659_amd.synth import make_workload
    w = make_workload(name, orders=orders)
    S = 16
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])
    mask = np.zeros((len(orders), len(w.cand)), np.uint8)
    mask[:, ::7] = 1
    r = oracle.score_lex(w.problem, w.intervals, w.cand, cs, ts, tile_mask=mask, n_threads=8)
    m = oracle.score(w.problem, w.intervals, w.cand, cs, ts, tile_mask=mask, dump=False, n_threads=8)
    sel = mask.astype(bool)
    np.testing.assert_array_equal(r.score_mm[sel], m.score[sel])
    np.testing.assert_array_equal(r.gap_mm, m.gap_now)
    meas = w.intervals.measured[:, w.cand].astype(bool)
    assert (r.score_mm[meas & sel] == 0).all() and (r.score_gp[meas & sel] == 0).all()
    for o in range(len(orders)):
        assert r.best[o] < 0 or not meas[o, r.best[o]]
