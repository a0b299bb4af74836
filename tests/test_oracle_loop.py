"""Pins of the profiling-loop oracle (Algorithm 1): hand-derived
trajectories on the HW3 instance (tests/golden/hw4_profile_loop.json) and
properties that hold on any workload whose hidden truth lies inside the
initial intervals:
  * a certified-feasible trajectory has 0 <= regret <= eps (its committed
    cells are measured, so its conservative value is its true value, and the
    optimistic value bounds the true optimum);
  * GPU-seconds are 300 s x TP summed over the revealed cells;
  * a fixed reveal order reveals the initially unmeasured candidates in that
    order;
  * with eps < 0 nothing certifies and every unmeasured candidate is revealed
    exactly once."""
import os

import numpy as np
import pytest

import oracle
from conftest import load_golden
from paper_2608_19659_amd.synth import Intervals, Problem, make_workload

STATES = {"UNDECIDED": oracle.UNDECIDED, "CERTIFIED_FEASIBLE": oracle.CERTIFIED_FEASIBLE,
          "CERTIFIED_INFEASIBLE": oracle.CERTIFIED_INFEASIBLE}
THREADS = min(os.cpu_count() or 1, 8)


def _intervals(d):
    return Intervals(*(np.array([d[k]], np.float32) for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi")),
                     np.array([d["measured"]], np.uint8))


@pytest.mark.parametrize("case", range(len(load_golden("hw4_profile_loop.json")["cases"])))
def test_hand_derived_trajectories(case):
    g = load_golden("hw4_profile_loop.json")
    c = g["cases"][case]
    floor = None if "floor" not in c else np.array(c["floor"], np.float32)
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"],
                floor_rps=floor)
    iv = _intervals(c.get("intervals", g["intervals"]))
    policy = oracle.POLICY_ORDER if c["policy"] == "order" else oracle.POLICY_SCORE
    r = oracle.profile_loop(p, iv, [c["truth_cap"]], [c["truth_tail"]], c.get("cand", g["cand"]),
                            np.array([c.get("cap_s", g["cap_s"])], np.float32),
                            np.array([c.get("tail_s", g["tail_s"])], np.float32),
                            eps=c["eps"], policy=policy, order=[c.get("order")], max_rounds=c.get("max_rounds"))
    assert r.state[0] == STATES[c["state"]], c["what"]
    assert r.finished[0] == c["finished"]
    assert r.rounds[0] == c["rounds"]
    assert list(r.reveals[0][: r.rounds[0]]) == c["reveals"]
    assert np.all(r.reveals[0][r.rounds[0]:] == -1)
    assert r.gpu_seconds[0] == c["gpu_seconds"]
    if "final_replicas" in c:
        assert r.final[0].tp_index == c["final_tp_index"] and r.final[0].replicas == c["final_replicas"]
        assert r.final[0].tau == c["final_tau"]
        assert r.tau_truth[0] == np.float32(c["tau_truth"]) and r.tau_oracle[0] == np.float32(c["tau_oracle"])
        assert r.regret[0] == c["regret"]


def _loop_inputs(name, orders, S):
    w = make_workload(name, orders=orders)
    O = len(orders)
    truth_cap = np.repeat(w.truth_cap[None], O, axis=0)
    truth_tail = np.repeat(w.truth_tail[None], O, axis=0)
    return w, truth_cap, truth_tail, w.cap_s[:, :, :S], w.tail_s[:, :, :S]


def _check_bookkeeping(w, r):
    p = w.problem
    tp_of = lambda cell: int(p.tp[(cell // p.n_levels) % p.n_tp])
    for o in range(len(r.rounds)):
        rev = [int(e) for e in r.reveals[o][: r.rounds[o]]]
        assert np.all(r.reveals[o][r.rounds[o]:] == -1)
        assert len(set(rev)) == len(rev)
        assert all(not w.intervals.measured[o, w.cand[e]] for e in rev)
        assert r.gpu_seconds[o] == sum(oracle.CELL_SECONDS * tp_of(int(w.cand[e])) for e in rev)
        assert r.regret[o] >= 0.0
        if r.state[o] == oracle.CERTIFIED_FEASIBLE:
            assert r.finished[o] == 1 and r.regret[o] <= 0.05


@pytest.mark.parametrize("name,orders,S", [("tiny-2class-G16", [0], 64),
                                          ("paper-shaped-2class-G16", [0, 1, 2, 3], 64)])
def test_score_policy_properties(name, orders, S):
    w, tc, tt, cs, ts = _loop_inputs(name, orders, S)
    r = oracle.profile_loop(w.problem, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, n_threads=THREADS)
    _check_bookkeeping(w, r)
    assert np.all(r.finished == 1)


def test_order_policy_follows_the_order():
    w, tc, tt, cs, ts = _loop_inputs("paper-shaped-2class-G16", [0, 1, 2, 3], 16)
    rng = np.random.default_rng(5)
    order = [rng.permutation(len(w.cand)) for _ in range(4)]
    r = oracle.profile_loop(w.problem, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05,
                            policy=oracle.POLICY_ORDER, order=order)
    _check_bookkeeping(w, r)
    for o in range(4):
        todo = [int(e) for e in order[o] if not w.intervals.measured[o, w.cand[e]]]
        assert list(r.reveals[o][: r.rounds[o]]) == todo[: r.rounds[o]]


def test_negative_eps_reveals_everything():
    w, tc, tt, cs, ts = _loop_inputs("paper-shaped-2class-G16", [0, 1], 16)
    r = oracle.profile_loop(w.problem, w.intervals, tc, tt, w.cand, cs, ts, eps=-1.0, n_threads=THREADS)
    _check_bookkeeping(w, r)
    for o in range(2):
        todo = {int(e) for e in range(len(w.cand)) if not w.intervals.measured[o, w.cand[e]]}
        assert r.state[o] == oracle.UNDECIDED and r.finished[o] == 1
        assert set(int(e) for e in r.reveals[o][: r.rounds[o]]) == todo
