"""Parity of the profiling loop (fs_profile_loop, Algorithm 1) with the
loop oracle: every trajectory's certificate state, end reason, reveal
sequence, GPU-seconds, returned allocation and its value on the true table,
element by element.  Covers the hand-derived trajectories, both reveal
policies, critical floors (the wave-per-scenario scorer), trajectories that
reveal every candidate, the round limit and the early-exit checks."""
import sys

import numpy as np
import pytest

import oracle
from conftest import load_golden
from paper_2608_19659_amd.synth import Intervals, Problem, make_workload

pytestmark = pytest.mark.gpu
STATES = {"UNDECIDED": 0, "CERTIFIED_FEASIBLE": 1, "CERTIFIED_INFEASIBLE": 2}


def note(msg):
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_2608_19659_amd import fleetsieve as fs
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    return torch, fs, fs.Context(0)


def gpu_loop(env, problem, iv, truth_cap, truth_tail, cand, cap_s, tail_s, eps, policy, order=None,
             max_rounds=None, check_every=4):
    torch, fs, ctx = env
    dev = "cuda:0"
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    r = fs.profile_loop(ctx, problem, fs.DeviceIntervals.from_host(iv, dev), t(np.asarray(truth_cap, np.float32)),
                        t(np.asarray(truth_tail, np.float32)), t(np.asarray(cand, np.int32)),
                        t(np.asarray(cap_s, np.float32)), t(np.asarray(tail_s, np.float32)), eps=eps,
                        policy=policy, order=None if order is None else t(np.asarray(order, np.int32)),
                        max_rounds=max_rounds, check_every=check_every)
    torch.cuda.synchronize()
    c = lambda x: x.cpu().numpy()
    return dict(state=c(r.state), finished=c(r.finished), rounds=c(r.rounds), gpu_seconds=c(r.gpu_seconds),
                reveals=c(r.reveals), objective=c(r.final["objective"]), tp_index=c(r.final["tp_index"]),
                replicas=c(r.final["replicas"]).view(np.uint16), tau_truth=c(r.tau_truth),
                tau_oracle=c(r.tau_oracle))


def assert_loop_equal(g, o, what=""):
    np.testing.assert_array_equal(g["state"], o.state, err_msg=what)
    np.testing.assert_array_equal(g["finished"], o.finished, err_msg=what)
    np.testing.assert_array_equal(g["rounds"], o.rounds, err_msg=what)
    np.testing.assert_array_equal(g["reveals"], o.reveals, err_msg=what)
    np.testing.assert_array_equal(g["gpu_seconds"], o.gpu_seconds, err_msg=what)
    for j, a in enumerate(o.final):
        assert g["objective"][j].view(np.uint32) == np.float32(a.tau).view(np.uint32), (what, j)
        assert list(g["tp_index"][j]) == [255 if t < 0 else t for t in a.tp_index], (what, j)
        assert list(g["replicas"][j]) == a.replicas, (what, j)
    np.testing.assert_array_equal(g["tau_truth"], o.tau_truth, err_msg=what)
    np.testing.assert_array_equal(g["tau_oracle"], o.tau_oracle, err_msg=what)


@pytest.mark.parametrize("case", range(len(load_golden("hw4_profile_loop.json")["cases"])))
def test_hand_derived_trajectories_on_gpu(env, case):
    g = load_golden("hw4_profile_loop.json")
    c = g["cases"][case]
    note(f"loop golden case {case}: {c['what']}")
    floor = None if "floor" not in c else np.array(c["floor"], np.float32)
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"],
                floor_rps=floor)
    d = c.get("intervals", g["intervals"])
    iv = Intervals(*(np.array([d[k]], np.float32) for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi")),
                   np.array([d["measured"]], np.uint8))
    policy = 1 if c["policy"] == "order" else 0
    order = None if policy == 0 else [c["order"]]
    r = gpu_loop(env, p, iv, [c["truth_cap"]], [c["truth_tail"]], c.get("cand", g["cand"]),
                 [c.get("cap_s", g["cap_s"])], [c.get("tail_s", g["tail_s"])], c["eps"], policy, order,
                 c.get("max_rounds"))
    assert r["state"][0] == STATES[c["state"]]
    assert r["finished"][0] == c["finished"] and r["rounds"][0] == c["rounds"]
    assert list(r["reveals"][0][: c["rounds"]]) == c["reveals"]
    assert r["gpu_seconds"][0] == c["gpu_seconds"]
    if "final_replicas" in c:
        assert list(r["replicas"][0]) == c["final_replicas"]
        assert list(r["tp_index"][0]) == [255 if t < 0 else t for t in c["final_tp_index"]]
        assert r["objective"][0] == np.float32(c["final_tau"])
        assert r["tau_truth"][0] == np.float32(c["tau_truth"]) and r["tau_oracle"][0] == np.float32(c["tau_oracle"])


def _inputs(name, orders, S, floors=None):
    w = make_workload(name, orders=orders)
    p = w.problem
    if floors is not None:
        p = Problem(p.tp, p.levels, p.demand, p.slo, p.budget, floor_rps=np.asarray(floors, np.float32))
    O = len(orders)
    tc = np.repeat(w.truth_cap[None], O, axis=0)
    tt = np.repeat(w.truth_tail[None], O, axis=0)
    return w, p, tc, tt, np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])


@pytest.mark.parametrize("name,orders,S,max_rounds", [
    ("tiny-2class-G16", [0], 64, None),
    ("paper-shaped-2class-G16", list(range(8)), 64, None),
    ("4class-G64", [1, 2], 256, 12),
    ("8class-G256", [0], 64, 4),
])
def test_score_policy_matches_oracle(env, name, orders, S, max_rounds):
    w, p, tc, tt, cs, ts = _inputs(name, orders, S)
    note(f"loop {name} orders={orders} S={S} score policy")
    o = oracle.profile_loop(p, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, max_rounds=max_rounds, n_threads=8)
    g = gpu_loop(env, p, w.intervals, tc, tt, w.cand, cs, ts, 0.05, 0, max_rounds=max_rounds)
    assert_loop_equal(g, o, name)


def test_order_policy_matches_oracle(env):
    w, p, tc, tt, cs, ts = _inputs("paper-shaped-2class-G16", list(range(8)), 16)
    rng = np.random.default_rng(11)
    order = np.stack([rng.permutation(len(w.cand)) for _ in range(8)]).astype(np.int32)
    note("loop paper-shaped order policy")
    o = oracle.profile_loop(p, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, policy=oracle.POLICY_ORDER,
                            order=order)
    g = gpu_loop(env, p, w.intervals, tc, tt, w.cand, cs, ts, 0.05, 1, order=order)
    assert_loop_equal(g, o, "order")


def test_floors_and_exhaustion_match_oracle(env):
    w, p, tc, tt, cs, ts = _inputs("paper-shaped-2class-G16", [0, 1, 2, 3], 32, floors=[1.0, 0.0])
    note("loop paper-shaped with a critical floor")
    o = oracle.profile_loop(p, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, n_threads=8)
    g = gpu_loop(env, p, w.intervals, tc, tt, w.cand, cs, ts, 0.05, 0)
    assert_loop_equal(g, o, "floors")
    w, p, tc, tt, cs, ts = _inputs("paper-shaped-2class-G16", [0, 1], 16)
    note("loop paper-shaped eps=-1 (every candidate revealed)")
    o = oracle.profile_loop(p, w.intervals, tc, tt, w.cand, cs, ts, eps=-1.0, n_threads=8)
    g = gpu_loop(env, p, w.intervals, tc, tt, w.cand, cs, ts, -1.0, 0)
    assert_loop_equal(g, o, "exhaustion")
    # candidates a subset of the cells (8 of 24): at exhaustion the loop
    # returns the best allocation over measured cells only
    w, p, tc, tt, cs, ts = _inputs("tiny-2class-G16", [0], 64)
    note("loop tiny-2class-G16 eps=-1 (candidate subset, exhaustion)")
    o = oracle.profile_loop(p, w.intervals, tc, tt, w.cand, cs, ts, eps=-1.0, n_threads=8)
    g = gpu_loop(env, p, w.intervals, tc, tt, w.cand, cs, ts, -1.0, 0)
    assert_loop_equal(g, o, "candidate subset")
    for name, rounds in (("tiny-2class-G16", 2), ("paper-shaped-2class-G16", 3)):
        w, p, tc, tt, cs, ts = _inputs(name, [0, 1] if name != "tiny-2class-G16" else [0], 16)
        note(f"loop {name} round limit {rounds}")
        o = oracle.profile_loop(p, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, max_rounds=rounds, n_threads=8)
        g = gpu_loop(env, p, w.intervals, tc, tt, w.cand, cs, ts, 0.05, 0, max_rounds=rounds)
        assert_loop_equal(g, o, f"round limit {name}")


def test_early_exit_checks_do_not_change_results(env):
    w, p, tc, tt, cs, ts = _inputs("paper-shaped-2class-G16", list(range(6)), 32)
    res = []
    for check_every in (0, 1, 5):
        note(f"loop check_every={check_every}")
        res.append(gpu_loop(env, p, w.intervals, tc, tt, w.cand, cs, ts, 0.05, 0, check_every=check_every))
    for r in res[1:]:
        for k in res[0]:
            np.testing.assert_array_equal(r[k], res[0][k], err_msg=k)


def test_oversized_loop_is_rejected_before_any_launch(env):
    """The exclusion scorer's work list indexes (order, candidate) pairs in
    int32: 65535 orders x 65535 candidates is rejected with
    FS_ERR_UNSUPPORTED by the host checks, before the pointer checks (every
    device pointer here is NULL, so nothing could be launched)."""
    import ctypes
    torch, fs, ctx = env
    lib = fs.load_library()
    p = Problem(tp=[1, 2, 4, 8], levels=[0.5, 1.0, 2.0], demand=[4.0, 2.0], slo=[30.0, 30.0], budget=16)
    ref = fs._ProblemRef(p)
    note("oversized loop rejected")
    st = lib.fs_profile_loop(ctx.handle, ref.ptr, fs._Intervals(), 65535, None, None, None, 65535, None, None, 64,
                             ctypes.c_float(0.05), fs.POLICY_SCORE, None, 4, 0, fs._LoopOut(), None, 0, None)
    assert st == fs.FS_ERR_UNSUPPORTED, lib.fs_last_error()
    assert b"2^31" in lib.fs_last_error()
    # the same sizes under a fixed reveal order never score, so the limit does not apply: the
    # NULL arrays are then what is rejected
    st = lib.fs_profile_loop(ctx.handle, ref.ptr, fs._Intervals(), 65535, None, None, None, 65535, None, None, 64,
                             ctypes.c_float(0.05), fs.POLICY_ORDER, None, 4, 0, fs._LoopOut(), None, 0, None)
    assert st == fs.FS_ERR_INVALID_ARGUMENT
