"""Oracle self-consistency and properties fixed by the mathematics:
three independent solvers agree, greedy water-filling (the textbook optimum
for max-min with nondecreasing utilities) matches the DP at large budgets,
and the invariants of the realisations (Section 4.1) hold."""
import math

import numpy as np
import pytest

from paper_2608_19659_amd.synth import Intervals, Problem, make_workload, random_point_tables, random_problem

TP_SETS = [[1, 2, 4, 8], [2, 4, 8], [1], [1, 3, 5], [2, 4]]


def _same_alloc(a, b):
    return (a.tau == b.tau and a.floors_met == b.floors_met and a.tp_index == b.tp_index
            and a.replicas == b.replicas and a.gpus == b.gpus and a.goodput == b.goodput)


@pytest.mark.parametrize("critical", [False, True])
@pytest.mark.parametrize("K", [1, 2, 3])
def test_brute_dp_threshold_agree(orc, K, critical):
    rng = np.random.default_rng(100 + K + 10 * critical)
    n_checked = 0
    for inst in range(300 if K < 3 else 120):
        tp = TP_SETS[inst % len(TP_SETS)]
        G = int(rng.integers(max(tp[0], 1), 17 if K < 3 else 13))
        p = random_problem(seed=inst * 7 + K, K=K, tp=tp, G=G, n_levels=int(rng.integers(1, 5)),
                           critical=critical)
        cap, tail = random_point_tables(p, 4, seed=inst + 1000 * K, cap_range=(0.0, 3.0),
                                        tail_range=(5.0, 45.0))
        for j in range(cap.shape[0]):
            a = orc.solve(p, cap[j], tail[j], "brute")
            d = orc.solve(p, cap[j], tail[j], "dp")
            t = orc.solve(p, cap[j], tail[j], "threshold")
            assert _same_alloc(a, d), (inst, j, a, d)
            assert t.tau == d.tau and t.floors_met == d.floors_met, (inst, j, t, d)
            n_checked += 1
    assert n_checked > 400


def _greedy_waterfill(caps, demand, t, G):
    """Max-min by repeatedly adding a replica to the currently worst class:
    optimal when every class's fulfillment is nondecreasing in its replica
    count.  Fulfillment is recomputed here with numpy binary32."""
    K = len(caps)
    r = np.zeros(K, dtype=np.int64)

    def f(i, n):
        if n == 0:
            return np.float32(0.0)
        q = np.float32(np.float32(n) * np.float32(caps[i])) / np.float32(demand[i])
        return min(np.float32(1.0), q)

    used = 0
    while used + t <= G:
        vals = [f(i, r[i]) for i in range(K)]
        i = int(np.argmin(vals))
        r[i] += 1
        used += t
    return min(f(i, r[i]) for i in range(K))


@pytest.mark.parametrize("K,t,G", [(16, 1, 1024), (8, 2, 512), (5, 4, 4096), (3, 1, 7), (12, 8, 1000)])
def test_dp_matches_waterfilling(orc, K, t, G):
    rng = np.random.default_rng(K * 1000 + G)
    for trial in range(3):
        caps = (np.rint(rng.uniform(0.05, 3.0, size=K) * 64) / 64).astype(np.float32)
        demand = rng.uniform(1.0, 200.0 if G >= 512 else 10.0, size=K).astype(np.float32)
        p = Problem(tp=[t], levels=[1.0e6], demand=demand, slo=np.full(K, 30.0), budget=G)
        cap = np.repeat(caps, 1).astype(np.float32)   # one TP, one level: one cell per class
        tail = np.full(K, 10.0, np.float32)
        d = orc.solve(p, cap, tail, "dp")
        th = orc.solve(p, cap, tail, "threshold")
        assert d.tau == _greedy_waterfill(caps, demand, t, G)
        assert th.tau == d.tau
        assert d.gpus <= G


def test_monotone_in_capacity_tail_and_budget(orc):
    """tau* is nondecreasing in every capacity and in G, nonincreasing in
    every tail (every option's fulfillment is, and max/min are monotone)."""
    rng = np.random.default_rng(7)
    for inst in range(40):
        p = random_problem(seed=500 + inst, K=3, tp=[1, 2, 4, 8], G=int(rng.integers(4, 20)), n_levels=3)
        cap, tail = random_point_tables(p, 1, seed=inst, cap_range=(0.0, 3.0), tail_range=(5.0, 45.0))
        cap, tail = cap[0], tail[0]
        base = orc.solve(p, cap, tail).tau
        c = int(rng.integers(p.n_cells))
        up = cap.copy(); up[c] += np.float32(0.5)
        assert orc.solve(p, up, tail).tau >= base
        tl = tail.copy(); tl[c] += np.float32(20.0)
        assert orc.solve(p, cap, tl).tau <= base
        p2 = Problem(p.tp, p.levels, p.demand, p.slo, p.budget + 3)
        assert orc.solve(p2, cap, tail).tau >= base


def test_class_permutation(orc):
    rng = np.random.default_rng(11)
    for inst in range(30):
        p = random_problem(seed=900 + inst, K=3, tp=[1, 2, 4, 8], G=14, n_levels=2)
        cap, tail = random_point_tables(p, 1, seed=inst, cap_range=(0.0, 3.0), tail_range=(5.0, 45.0))
        perm = rng.permutation(3)
        q = Problem(p.tp, p.levels, p.demand[perm], p.slo[perm], p.budget)
        per = p.n_tp * p.n_levels
        cells = np.concatenate([np.arange(i * per, (i + 1) * per) for i in perm])
        a = orc.solve(p, cap[0], tail[0])
        b = orc.solve(q, cap[0][cells], tail[0][cells])
        assert a.tau == b.tau
        assert [a.tp_index[i] for i in perm] == b.tp_index
        assert [a.replicas[i] for i in perm] == b.replicas


def test_pairwise_sum_order(orc):
    # Exactly representable values: every order gives the exact sum.
    x = np.arange(1, 1001, dtype=np.float64) / 64.0
    assert orc.pairwise_sum(x) == math.fsum(x)
    # The association is the pairwise tree, not left-to-right:
    # (1e16 + 1) + (-1e16 + 1) = 1e16 + (-1e16) = 0, while sequential gives 1.
    assert orc.pairwise_sum([1e16, 1.0, -1e16, 1.0]) == 0.0
    # Zero padding to a power of two: [a, b, c] -> (a + b) + (c + 0).
    assert orc.pairwise_sum([1e16, 1.0, 1.0]) == (1e16 + 1.0) + 1.0


def test_invariants_on_paper_shaped_workload(orc):
    """tau- <= tau+, 0 <= Gamma(o,e,s) <= Gamma_t, score in [0, Gamma_t] and a
    measured candidate scores exactly 0 (samples lie inside the intervals)."""
    w = make_workload("paper-shaped-2class-G16", orders=[0, 1, 2, 3])
    E = w.n_cand
    mask = np.zeros((w.n_orders, E), np.uint8)
    mask[:, ::6] = 1
    r = orc.score(w.problem, w.intervals, w.cand, w.cap_s, w.tail_s, tile_mask=mask, n_threads=8)
    for o in range(w.n_orders):
        for e in np.nonzero(mask[o])[0]:
            tm, tp = r.tau_dump[o, e, :, 0], r.tau_dump[o, e, :, 1]
            assert np.all(tm <= tp)
            gam = tp.astype(np.float64) - tm.astype(np.float64)
            assert np.all(gam >= 0) and np.all(gam <= r.gap_now[o])
            assert 0.0 <= r.score[o, e] <= r.gap_now[o]
            if w.intervals.measured[o, w.cand[e]]:
                assert r.score[o, e] == 0.0


def test_point_intervals_give_zero_scores(orc):
    w = make_workload("tiny-2class-G16")
    tc, tt = w.truth_cap[None], w.truth_tail[None]
    iv = Intervals(tc, tc, tt, tt, np.zeros_like(w.intervals.measured))
    cs = np.broadcast_to(w.truth_cap[w.cand][None, :, None], w.cap_s.shape).copy()
    ts = np.broadcast_to(w.truth_tail[w.cand][None, :, None], w.tail_s.shape).copy()
    r = orc.score(w.problem, iv, w.cand, cs, ts)
    assert r.gap_now[0] == 0.0
    assert np.all(r.score == 0.0)


@pytest.mark.parametrize("name,n_orders", [("paper-shaped-2class-G16", 24), ("4class-G64", 6)])
def test_health_gates(orc, name, n_orders):
    """The synthetic workloads are not degenerate: at least 30% of orders have
    an open gap, every such order has a candidate with a positive score (there
    is something decision-critical to measure), and at least 1% of all
    scenarios close part of the gap."""
    w = make_workload(name, orders=list(range(n_orders)))
    S = 16
    r = orc.score(w.problem, w.intervals, w.cand, w.cap_s[:, :, :S], w.tail_s[:, :, :S],
                  n_threads=8)
    open_gap = r.gap_now > 0
    assert np.mean(open_gap) >= 0.30
    assert np.all(np.any(r.score[open_gap] > 0, axis=1))
    gam = r.tau_dump[..., 1].astype(np.float64) - r.tau_dump[..., 0]
    assert np.mean(gam < r.gap_now[:, None, None]) >= 0.01
