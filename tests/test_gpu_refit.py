"""The interval refit (Algorithm 1's fit step, fs_refit_intervals) and the
profiling loop with it, on the GPU through the C ABI, against the
hand-derived case and the oracle bit for bit."""
import ctypes
import sys

import numpy as np
import pytest

import oracle
from conftest import load_golden
from paper_2608_19659_amd.synth import Intervals, Problem, make_workload
from test_oracle_refit import _iv, _random_state

pytestmark = pytest.mark.gpu


def note(msg):
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_2608_19659_amd import fleetsieve as fs
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    return torch, fs, fs.Context(0)


def _t(env, a):
    return env[0].from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def gpu_refit(env, p, iv):
    torch, fs, ctx = env
    r = fs.refit_intervals(ctx, p, fs.DeviceIntervals.from_host(iv, "cuda:0"))
    torch.cuda.synchronize()
    return {k: getattr(r, k).cpu().numpy() for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi")}


def assert_same(got, want, what=""):
    for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi"):
        np.testing.assert_array_equal(got[k].view(np.uint32), np.asarray(getattr(want, k), np.float32).view(np.uint32),
                                      err_msg=f"{what} {k}")


def test_hand_derived_case_on_gpu(env):
    g = load_golden("refit.json")
    note("refit golden case")
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"])
    r = gpu_refit(env, p, _iv(g["before"]))
    for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi"):
        assert list(r[k][0]) == g["after"][k], k


@pytest.mark.parametrize("name,seed,frac", [("paper-shaped-2class-G16", 1, 0.3), ("4class-G64", 2, 0.5),
                                            ("16class-G1024", 3, 0.4), ("paper-shaped-2class-G16-knee", 4, 0.3),
                                            ("4class-G64-knee", 5, 0.2), ("4class-G64", 6, 0.0),
                                            ("4class-G64", 7, 1.0)])
def test_refit_matches_oracle(env, name, seed, frac):
    w, iv = _random_state(name, seed, frac)
    note(f"refit {name} seed {seed} measured fraction {frac}")
    assert_same(gpu_refit(env, w.problem, iv), oracle.refit_intervals(w.problem, iv), name)


def test_round_down_and_in_place(env):
    """A bound binary32 cannot hold (TP {1, 3, 9}) is rounded down as in the
    oracle; outputs aliasing the inputs give the same result."""
    torch, fs, ctx = env
    p = Problem(tp=[1, 3, 9], levels=[1.0], demand=[1.0], slo=[30.0], budget=9)
    iv = _iv({"cap_lo": [1.0, 0.1, 1.0], "cap_hi": [1.0, 5.0, 1.0], "tail_lo": [1.0] * 3, "tail_hi": [1.0] * 3,
              "measured": [1, 0, 1]})
    note("refit round-down case and in-place refit")
    assert_same(gpu_refit(env, p, iv), oracle.refit_intervals(p, iv), "round down")
    w, iv2 = _random_state("4class-G64-knee", 9, 0.3)
    d = fs.DeviceIntervals.from_host(iv2, "cuda:0")
    ref = fs._ProblemRef(w.problem)
    O = d.cap_lo.shape[0]
    fs._check(fs.load_library().fs_refit_intervals(ctx.handle, ref.ptr, fs._intervals_struct(d, O, ref.N), O,
                                                   d.cap_lo.data_ptr(), d.tail_lo.data_ptr(), d.tail_hi.data_ptr(),
                                                   fs._stream(d.cap_lo.device, None)))
    torch.cuda.synchronize()
    got = {k: getattr(d, k).cpu().numpy() for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi")}
    assert_same(got, oracle.refit_intervals(w.problem, iv2), "in place")


@pytest.mark.parametrize("name,orders,S,max_rounds,objective", [
    ("paper-shaped-2class-G16-knee", list(range(8)), 64, None, "maxmin"),
    ("4class-G64-knee", [0, 1, 2, 3], 128, 12, "maxmin"),
    ("paper-shaped-2class-G16-knee", list(range(8, 14)), 32, None, "lex"),
])
def test_loop_with_refit_matches_oracle(env, name, orders, S, max_rounds, objective):
    torch, fs, ctx = env
    w = make_workload(name, orders=orders)
    O = len(orders)
    tc = np.repeat(w.truth_cap[None], O, axis=0)
    tt = np.repeat(w.truth_tail[None], O, axis=0)
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])
    note(f"loop with refit {name} orders={orders} S={S} {objective}")
    o = oracle.profile_loop(w.problem, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, max_rounds=max_rounds,
                            n_threads=8, objective=objective, refit=True)
    ctx.set_option(fs.OPT_LOOP_OBJECTIVE, fs.OBJECTIVE_LEXICOGRAPHIC if objective == "lex" else fs.OBJECTIVE_MAXMIN)
    try:
        r = fs.profile_loop(ctx, w.problem, fs.DeviceIntervals.from_host(w.intervals, "cuda:0"), _t(env, tc),
                            _t(env, tt), _t(env, w.cand), _t(env, cs), _t(env, ts), eps=0.05, max_rounds=max_rounds,
                            refit=True)
        torch.cuda.synchronize()
    finally:
        ctx.set_option(fs.OPT_LOOP_OBJECTIVE, fs.OBJECTIVE_MAXMIN)
        ctx.set_option(fs.OPT_LOOP_REFIT, 0)
    np.testing.assert_array_equal(r.state.cpu().numpy(), o.state)
    np.testing.assert_array_equal(r.rounds.cpu().numpy(), o.rounds)
    np.testing.assert_array_equal(r.reveals.cpu().numpy(), o.reveals)
    np.testing.assert_array_equal(r.gpu_seconds.cpu().numpy(), o.gpu_seconds)
    np.testing.assert_array_equal(r.tau_truth.cpu().numpy(), o.tau_truth)
    reps = r.final["replicas"].cpu().numpy()
    for j, a in enumerate(o.final):
        assert list(reps[j].view(np.uint16)) == a.replicas, j


def gpu_clamp(env, p, iv, cand, cs, ts):
    torch, fs, ctx = env
    c, t = fs.clamp_samples(ctx, p, fs.DeviceIntervals.from_host(iv, "cuda:0"),
                            _t(env, np.asarray(cand, np.int32)), _t(env, cs), _t(env, ts))
    torch.cuda.synchronize()
    return c.cpu().numpy(), t.cpu().numpy()


def test_clamp_hand_derived_on_gpu(env):
    """fs_refit_intervals then fs_clamp_samples on the hand-derived case
    (tests/golden/clamp_samples.json): the samples land in the refitted
    intervals, exactly at the bounds where they fall outside."""
    g = load_golden("clamp_samples.json")
    note("clamp golden case")
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"])
    r = gpu_refit(env, p, _iv(g["intervals"]))
    for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi"):
        assert list(r[k][0]) == g["refit"][k], k
    f = Intervals(r["cap_lo"], r["cap_hi"], r["tail_lo"], r["tail_hi"], _iv(g["intervals"]).measured)
    c, t = gpu_clamp(env, p, f, g["cand"], np.array([g["cap_s"]], np.float32), np.array([g["tail_s"]], np.float32))
    assert c.tolist() == [g["clamped_cap_s"]] and t.tolist() == [g["clamped_tail_s"]]


@pytest.mark.parametrize("name,seed,frac,S", [("4class-G64-knee", 3, 0.3, 4096), ("paper-shaped-2class-G16", 1, 0.3, 1000),
                                              ("16class-G1024", 2, 0.4, 256)])
def test_clamp_matches_oracle(env, name, seed, frac, S):
    """k_clamp_samples against oracle.clamp_samples, bit for bit, on the
    refit of a random measured state (ragged S included)."""
    w0, iv = _random_state(name, seed, frac)
    w = make_workload(name, orders=list(range(4)))
    note(f"clamp {name} S={S}")
    f = oracle.refit_intervals(w.problem, iv)
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])
    want_c, want_t = oracle.clamp_samples(f, w.cand, cs, ts)
    got_c, got_t = gpu_clamp(env, w.problem, f, w.cand, cs, ts)
    np.testing.assert_array_equal(got_c.view(np.uint32), want_c.view(np.uint32))
    np.testing.assert_array_equal(got_t.view(np.uint32), want_t.view(np.uint32))
    assert (want_c != cs).any() or (want_t != ts).any()


@pytest.mark.parametrize("case", range(2))
def test_fit_step_saves_a_reveal_on_gpu(env, case):
    """The hand-derived loop of tests/golden/refit_loop.json on the GPU:
    with the fit step the refitted tail closes the gap and the loop
    certifies with no reveal; without it one reveal is paid."""
    torch, fs, ctx = env
    g = load_golden("refit_loop.json")
    c = g["cases"][case]
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"])
    d = g["intervals"]
    iv = Intervals(*(np.array([d[k]], np.float32) for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi")),
                   np.array([d["measured"]], np.uint8))
    note(f"refit loop golden case refit={c['refit']}")
    try:
        r = fs.profile_loop(ctx, p, fs.DeviceIntervals.from_host(iv, "cuda:0"),
                            _t(env, np.array([g["truth_cap"]], np.float32)),
                            _t(env, np.array([g["truth_tail"]], np.float32)), _t(env, np.array(g["cand"], np.int32)),
                            _t(env, np.array([g["cap_s"]], np.float32)), _t(env, np.array([g["tail_s"]], np.float32)),
                            eps=g["eps"], refit=c["refit"])
        torch.cuda.synchronize()
    finally:
        ctx.set_option(fs.OPT_LOOP_REFIT, 0)
    assert int(r.state.cpu()[0]) == 1
    assert int(r.rounds.cpu()[0]) == c["rounds"]
    assert list(r.reveals.cpu().numpy()[0][: c["rounds"]]) == c["reveals"]
    assert float(r.gpu_seconds.cpu()[0]) == c["gpu_seconds"]
    assert list(r.final["tp_index"].cpu().numpy()[0]) == c["final_tp_index"]
    assert list(r.final["replicas"].cpu().numpy()[0].view(np.uint16)) == c["final_replicas"]
    assert float(r.final["objective"].cpu()[0]) == np.float32(c["final_tau"])
    assert float(r.tau_truth.cpu()[0]) == np.float32(c["tau_truth"])
