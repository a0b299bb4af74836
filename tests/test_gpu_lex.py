"""The whole lexicographic objective (Section 3, levels 1-4) and the
stage-wise certificate (Section 4.2) on the GPU, through the C ABI
(fs_solve_batch_lex, fs_certify_lex), against the hand-derived cases and
the oracle bit for bit: tau*, floors, allocation, binary32 goodput, level
(3)'s binary64 total, states and both gaps."""
import sys
from types import SimpleNamespace

import numpy as np
import pytest

import oracle
from conftest import load_golden
from paper_2608_19659_amd.synth import Intervals, Problem, make_workload, random_point_tables, random_problem
from test_oracle_lex import STATES, hw1_tables

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


def gpu_solve_lex(env, p, cap, tail):
    torch, fs, ctx = env
    out = fs.solve_batch_lex(ctx, p, _t(env, cap), _t(env, tail))
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def assert_lex_equal(p, g, j, a, what=""):
    assert g["objective"][j].view(np.uint32) == np.float32(a.tau).view(np.uint32), (what, g["objective"][j], a.tau)
    assert int(g["floors_met"][j]) == a.floors_met, what
    assert list(g["tp_index"][j]) == [255 if t < 0 else t for t in a.tp_index], (what, list(g["tp_index"][j]),
                                                                                 a.tp_index)
    assert list(g["replicas"][j].view(np.uint16)) == a.replicas, (what, a.replicas)
    assert g["goodput"][j].view(np.uint32) == np.float32(a.goodput).view(np.uint32), what
    assert g["goodput64"][j] == a.goodput64, (what, g["goodput64"][j], a.goodput64)


@pytest.mark.parametrize("case", range(len(load_golden("lex_objective.json")["solves"])))
def test_hand_derived_solves_on_gpu(env, case):
    g = load_golden("lex_objective.json")
    c = g["solves"][case]
    note(f"lex golden solve: {c['what']}")
    p, cap, tail = hw1_tables(g, c["budget"], c.get("floor"), c.get("code_tail"), c.get("tail_override", ()))
    r = gpu_solve_lex(env, p, cap[None], tail[None])
    assert r["objective"][0] == np.float32(c["tau"])
    assert [0 if t == 255 else int(p.tp[t]) for t in r["tp_index"][0]] == c["tp"]
    assert list(r["replicas"][0].view(np.uint16)) == c["replicas"]
    assert r["goodput64"][0] == c["goodput"] and r["goodput"][0] == np.float32(c["goodput"])


@pytest.mark.parametrize("case", range(len(load_golden("lex_objective.json")["certificates"])))
def test_hand_derived_certificates_on_gpu(env, case):
    torch, fs, ctx = env
    g = load_golden("lex_objective.json")
    c = g["certificates"][case]
    note(f"lex golden certificate: {c['what']}")
    p, cap, tail = hw1_tables(g, c["budget"])
    lo, hi = cap.copy(), cap.copy()
    lo[c["cell"]] = c["cap_lo"]
    if c["measured_cell"]:
        hi[c["cell"]] = c["cap_lo"]
    meas = np.ones(p.n_cells, np.uint8)
    meas[c["cell"]] = c["measured_cell"]
    iv = Intervals(lo[None], hi[None], tail[None], tail[None], meas[None])
    r = fs.certify_lex(ctx, p, fs.DeviceIntervals.from_host(iv, "cuda:0"), eps=c["eps"])
    torch.cuda.synchronize()
    assert r.state.item() == STATES[c["state"]]
    assert r.gap_maxmin.item() == c["gap_mm"]
    assert r.gap_goodput.item() == c["gap_gp_num"] / c["gap_gp_den"]
    cons_tp = [0 if t == 255 else int(p.tp[t]) for t in r.cons["tp_index"][0].cpu().numpy()]
    assert cons_tp == c["cons_tp"] and list(r.cons["replicas"][0].cpu().numpy()) == c["cons_replicas"]


@pytest.mark.parametrize("critical", [False, True])
def test_random_problems_match_oracle(env, critical):
    rng = np.random.default_rng(15 + critical)
    for inst in range(24):
        tp = [[1, 2, 4, 8], [2, 4, 8], [1], [1, 3, 5], [2, 4]][inst % 5]
        K = int(rng.integers(1, 6))
        G = int(rng.integers(tp[0], 40 if inst % 3 else 150))
        p = random_problem(seed=3000 + inst, K=K, tp=tp, G=G, n_levels=int(rng.integers(1, 6)), critical=critical)
        cap, tail = random_point_tables(p, 16, seed=inst, cap_range=(0.0, 3.0), tail_range=(5.0, 45.0))
        note(f"lex dense inst {inst} K={K} G={G} tp={tp} critical={critical}")
        g = gpu_solve_lex(env, p, cap, tail)
        for j in range(cap.shape[0]):
            assert_lex_equal(p, g, j, oracle.solve(p, cap[j], tail[j], "lex"), f"inst {inst} row {j}")


@pytest.mark.parametrize("name,n", [("paper-shaped-2class-G16", 64), ("4class-G64", 32), ("8class-G256", 8),
                                    ("16class-G1024", 2)])
def test_workload_realisations_match_oracle(env, name, n):
    """Both corners of the workloads' intervals, the 16-class G=1024 case at
    the largest budget the stage's LDS holds for it."""
    w = make_workload(name, orders=list(range(min(n, 4))), with_samples=False)
    p = w.problem
    iv = w.intervals
    cap = np.concatenate([iv.cap_lo, iv.cap_hi])[:n]
    tail = np.concatenate([iv.tail_hi, iv.tail_lo])[:n]
    note(f"lex dense {name} x {cap.shape[0]}")
    g = gpu_solve_lex(env, p, cap, tail)
    for j in range(cap.shape[0]):
        assert_lex_equal(p, g, j, oracle.solve(p, cap[j], tail[j], "lex"), f"{name} row {j}")


@pytest.mark.parametrize("name,orders", [("paper-shaped-2class-G16", list(range(12))), ("4class-G64", [0, 1, 2, 3]),
                                         ("8class-G256", [0, 1])])
def test_certificates_match_oracle(env, name, orders):
    torch, fs, ctx = env
    w = make_workload(name, orders=orders, with_samples=False)
    note(f"lex certify {name} orders={orders}")
    r = fs.certify_lex(ctx, w.problem, fs.DeviceIntervals.from_host(w.intervals, "cuda:0"), eps=0.05)
    torch.cuda.synchronize()
    o = oracle.certify_lex(w.problem, w.intervals, eps=0.05)
    np.testing.assert_array_equal(r.state.cpu().numpy(), o.state)
    np.testing.assert_array_equal(r.gap_maxmin.cpu().numpy(), o.gap_mm)
    np.testing.assert_array_equal(r.gap_goodput.cpu().numpy(), o.gap_gp)
    c = {k: v.cpu().numpy() for k, v in r.cons.items()}
    op = {k: v.cpu().numpy() for k, v in r.opt.items()}
    for j in range(len(orders)):
        for got, a in ((c, o.cons[j]), (op, o.opt[j])):
            assert list(got["tp_index"][j]) == [255 if t < 0 else t for t in a.tp_index], (name, j)
            assert list(got["replicas"][j].view(np.uint16)) == a.replicas, (name, j)
            assert got["goodput"][j].view(np.uint32) == np.float32(a.goodput).view(np.uint32), (name, j)
    assert (o.gap_gp > 0).any()


def test_unsupported_sizes_are_rejected(env):
    torch, fs, ctx = env
    p = random_problem(seed=5, K=64, tp=[1, 2, 4, 8], G=512, n_levels=2)
    note("lex K=64 G=512: rejected before any launch")
    cap = torch.zeros((1, p.n_cells), device="cuda:0")
    with pytest.raises(fs.FleetSieveError) as e:
        fs.solve_batch_lex(ctx, p, cap, cap)
    assert e.value.status == fs.FS_ERR_UNSUPPORTED


def _gpu_loop(env, p, iv, tc, tt, cand, cs, ts, eps, objective, max_rounds=None, kernel=0):
    torch, fs, ctx = env
    ctx.set_option(fs.OPT_LOOP_OBJECTIVE, objective)
    ctx.set_score_kernel(kernel)
    try:
        r = fs.profile_loop(ctx, p, fs.DeviceIntervals.from_host(iv, "cuda:0"), _t(env, tc), _t(env, tt),
                            _t(env, np.asarray(cand, np.int32)), _t(env, cs), _t(env, ts), eps=eps,
                            max_rounds=max_rounds)
        torch.cuda.synchronize()
    finally:
        ctx.set_option(fs.OPT_LOOP_OBJECTIVE, fs.OBJECTIVE_MAXMIN)
        ctx.set_score_kernel(0)
    return {k: (v.cpu().numpy() if hasattr(v, "cpu") else {kk: vv.cpu().numpy() for kk, vv in v.items()})
            for k, v in vars(r).items()}


@pytest.mark.parametrize("objective", ["lex", "maxmin"])
def test_hand_derived_loop_on_gpu(env, objective):
    from test_oracle_lex import _loop_inputs
    torch, fs, ctx = env
    g = load_golden("lex_objective.json")
    c = g["loop"]
    p, iv, tc, tt, cand, cs, ts = _loop_inputs(g, c)
    note(f"lex golden loop, {objective}")
    code = fs.OBJECTIVE_LEXICOGRAPHIC if objective == "lex" else fs.OBJECTIVE_MAXMIN
    r = _gpu_loop(env, p, iv, tc, tt, cand, cs, ts, c["eps"], code)
    want = c[objective]
    assert r["state"][0] == STATES[want["state"]] and r["rounds"][0] == want["rounds"]
    assert list(r["reveals"][0][: want["rounds"]]) == want["reveals"]
    assert r["gpu_seconds"][0] == want["gpu_seconds"]
    assert [0 if t == 255 else int(p.tp[t]) for t in r["final"]["tp_index"][0]] == want["final_tp"]
    assert list(r["final"]["replicas"][0].view(np.uint16)) == want["final_replicas"]
    assert r["tau_truth"][0] == np.float32(want["tau_truth"])


@pytest.mark.parametrize("kernel", [0, 1])
@pytest.mark.parametrize("name,orders,S,max_rounds", [("paper-shaped-2class-G16", list(range(8)), 64, None),
                                                      ("4class-G64", [1, 2], 8, 12), ("6class-G32", [0], 16, 8)])
def test_loop_under_whole_objective_matches_oracle(env, name, orders, S, max_rounds, kernel):
    torch, fs, ctx = env
    w = make_workload(name, orders=orders)
    O = len(orders)
    tc = np.repeat(w.truth_cap[None], O, axis=0)
    tt = np.repeat(w.truth_tail[None], O, axis=0)
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])
    note(f"lex loop {name} orders={orders} S={S} kernel={kernel}")
    o = oracle.profile_loop(w.problem, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, max_rounds=max_rounds,
                            n_threads=8, objective="lex")
    r = _gpu_loop(env, w.problem, w.intervals, tc, tt, w.cand, cs, ts, 0.05, fs.OBJECTIVE_LEXICOGRAPHIC,
                  max_rounds, kernel)
    np.testing.assert_array_equal(r["state"], o.state)
    np.testing.assert_array_equal(r["rounds"], o.rounds)
    np.testing.assert_array_equal(r["reveals"], o.reveals)
    np.testing.assert_array_equal(r["gpu_seconds"], o.gpu_seconds)
    np.testing.assert_array_equal(r["tau_truth"], o.tau_truth)
    for j, a in enumerate(o.final):
        assert list(r["final"]["replicas"][j].view(np.uint16)) == a.replicas, j
        assert list(r["final"]["tp_index"][j]) == [255 if t < 0 else t for t in a.tp_index], j


def test_hand_derived_stagewise_score_on_gpu(env):
    from test_oracle_lex import _score_inputs
    torch, fs, ctx = env
    g = load_golden("lex_objective.json")
    c = g["score"]
    p, iv, cand, cs, ts = _score_inputs(g, c)
    note("stage-wise score golden case")
    r = fs.score_candidates_lex(ctx, p, fs.DeviceIntervals.from_host(iv, "cuda:0"), _t(env, cand), _t(env, cs),
                                _t(env, ts))
    torch.cuda.synchronize()
    assert list(r.score_maxmin.cpu().numpy()[0]) == c["score_mm"]
    assert list(r.score_goodput.cpu().numpy()[0]) == [x / c["score_gp_den"] for x in c["score_gp_num"]]
    assert r.best.item() == c["best"]


def _score_lex(env, w, cs, ts, kernel=0):
    """The stage-wise score through the C ABI; kernel 1 solves every scenario
    in full, the default takes the goodput stage from per-interval tables
    where the problem allows it."""
    torch, fs, ctx = env
    div = fs.DeviceIntervals.from_host(w.intervals, "cuda:0")
    ctx.set_score_kernel(kernel)
    try:
        r = fs.score_candidates_lex(ctx, w.problem, div, _t(env, w.cand), _t(env, cs), _t(env, ts))
        torch.cuda.synchronize()
    finally:
        ctx.set_score_kernel(0)
    return {k: getattr(r, k).cpu().numpy() for k in ("score_maxmin", "score_goodput", "gap_maxmin", "gap_goodput",
                                                     "best")}


def _assert_score_lex_equal(g, o, what):
    np.testing.assert_array_equal(g["score_maxmin"], o.score_mm, err_msg=what)
    np.testing.assert_array_equal(g["score_goodput"], o.score_gp, err_msg=what)
    np.testing.assert_array_equal(g["gap_maxmin"], o.gap_mm, err_msg=what)
    np.testing.assert_array_equal(g["gap_goodput"], o.gap_gp, err_msg=what)
    np.testing.assert_array_equal(g["best"], o.best, err_msg=what)


@pytest.mark.parametrize("kernel", [0, 1])
@pytest.mark.parametrize("name,orders,S", [("paper-shaped-2class-G16", [0, 3, 5], 16), ("4class-G64", [1], 8),
                                           ("tiny-2class-G16", None, 65), ("6class-G32", [0, 1], 64),
                                           ("12class-G64", [2], 16), ("4class-G64", [0, 5], 130)])
def test_stagewise_score_matches_oracle(env, name, orders, S, kernel):
    """Both scorers (full solves, kernel 1; per-interval tables, the default)
    against the oracle bit for bit, with a ragged last chunk of samples where
    S is not a multiple of 64; the max-min stage also against the max-min
    scorer."""
    torch, fs, ctx = env
    w = make_workload(name, orders=orders)
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])
    note(f"stage-wise score {name} orders={orders} S={S} kernel={kernel}")
    g = _score_lex(env, w, cs, ts, kernel)
    m = fs.score_candidates(ctx, w.problem, fs.DeviceIntervals.from_host(w.intervals, "cuda:0"), _t(env, w.cand),
                            _t(env, cs), _t(env, ts))
    torch.cuda.synchronize()
    o = oracle.score_lex(w.problem, w.intervals, w.cand, cs, ts, n_threads=16)
    _assert_score_lex_equal(g, o, f"{name} kernel {kernel}")
    np.testing.assert_array_equal(g["score_maxmin"], m.score.cpu().numpy())


def test_stagewise_score_8class_matches_oracle(env):
    """8 classes, G = 256 (about 450 distinct option ratios per realisation):
    the per-interval tables against the oracle on one order."""
    w = make_workload("8class-G256", orders=[3])
    S = 4
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])
    note("stage-wise score 8class-G256 order 3 S=4")
    g = _score_lex(env, w, cs, ts)
    o = oracle.score_lex(w.problem, w.intervals, w.cand, cs, ts, n_threads=16)
    _assert_score_lex_equal(g, o, "8class-G256")


def test_stagewise_scorers_agree_at_bench_size(env):
    """The configuration the stage-wise score is timed on (4 classes, G = 64,
    16 orders, every cell a candidate, 64 samples): the per-interval tables
    against the full solves bit for bit, and the oracle on sampled tiles."""
    w = make_workload("4class-G64")
    S = 64
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])
    note("stage-wise score 4class-G64 all orders S=64: tables vs full solves")
    fast = _score_lex(env, w, cs, ts, 0)
    full = _score_lex(env, w, cs, ts, 1)
    for k in fast:
        np.testing.assert_array_equal(fast[k], full[k], err_msg=k)
    from paper_2608_19659_amd.synth import seeded_tiles, tile_mask
    tiles = seeded_tiles(w, 24, seed=77)
    o = oracle.score_lex(w.problem, w.intervals, w.cand, cs, ts, tile_mask=tile_mask(w, tiles), n_threads=16)
    for (oi, e) in tiles:
        assert fast["score_maxmin"][oi, e] == o.score_mm[oi, e], (oi, e)
        assert fast["score_goodput"][oi, e] == o.score_gp[oi, e], (oi, e)


def _random_score_inputs(p, O, S, seed, measured_frac=0.2):
    rng = np.random.default_rng(seed)
    N = p.n_cells
    lo = (np.rint(rng.uniform(0.0, 3.0, (O, N)) * 64) / 64).astype(np.float32)
    hi = (lo + np.rint(rng.uniform(0.0, 1.0, (O, N)) * 64) / 64).astype(np.float32)
    tl = rng.uniform(2.0, 50.0, (O, N)).astype(np.float32)
    th = (tl * rng.uniform(1.0, 1.6, (O, N))).astype(np.float32)
    meas = (rng.random((O, N)) < measured_frac).astype(np.uint8)
    hi = np.where(meas == 1, lo, hi).astype(np.float32)
    th = np.where(meas == 1, tl, th).astype(np.float32)
    cand = np.arange(N, dtype=np.int32)
    u = rng.uniform(0, 1, (O, N, S)).astype(np.float32)
    cs = (lo[:, :, None] + (hi - lo)[:, :, None] * u).astype(np.float32)
    ts = (tl[:, :, None] + (th - tl)[:, :, None] * rng.uniform(0, 1, (O, N, S))).astype(np.float32)
    return Intervals(lo, hi, tl, th, meas), cand, cs, ts


@pytest.mark.parametrize("kernel", [0, 1])
def test_stagewise_score_random_problems(env, kernel):
    """Random problems without floors (TP sets with odd degrees, a single
    class, budgets that are not powers of two, tails on both sides of the
    SLO, some revealed cells, S not a multiple of 64): both scorers against
    the oracle bit for bit."""
    rng = np.random.default_rng(41)
    for inst in range(16):
        tp = [[1, 2, 4, 8], [2, 4, 8], [1], [1, 3, 5], [2, 4]][inst % 5]
        K = int(rng.integers(1, 6))
        G = int(rng.integers(max(tp[0], 2), 90))
        p = random_problem(seed=5100 + inst, K=K, tp=tp, G=G, n_levels=int(rng.integers(1, 6)))
        O, S = int(rng.integers(1, 4)), int(rng.integers(1, 130))
        iv, cand, cs, ts = _random_score_inputs(p, O, S, seed=inst)
        note(f"stage-wise random inst {inst} K={K} G={G} tp={tp} O={O} S={S} kernel={kernel}")
        w = SimpleNamespace(problem=p, intervals=iv, cand=cand)
        g = _score_lex(env, w, cs, ts, kernel)
        o = oracle.score_lex(p, iv, cand, cs, ts, n_threads=16)
        _assert_score_lex_equal(g, o, f"inst {inst}")


@pytest.mark.parametrize("kernel", [0, 1])
def test_stagewise_score_many_tp_degrees(env, kernel):
    """Five to eight TP degrees (the interval tables compiled for eight):
    both scorers against the oracle bit for bit."""
    rng = np.random.default_rng(61)
    for inst in range(6):
        tp = [[1, 2, 4, 8, 16], [1, 2, 3, 4, 6, 8], [1, 2, 3, 4, 5, 6, 7, 8]][inst % 3]
        K = int(rng.integers(1, 5))
        G = int(rng.integers(tp[-1], 90))
        p = random_problem(seed=6100 + inst, K=K, tp=tp, G=G, n_levels=int(rng.integers(1, 5)))
        O, S = int(rng.integers(1, 3)), int(rng.integers(1, 100))
        iv, cand, cs, ts = _random_score_inputs(p, O, S, seed=60 + inst)
        note(f"stage-wise many TP degrees inst {inst} K={K} G={G} tp={tp} O={O} S={S} kernel={kernel}")
        w = SimpleNamespace(problem=p, intervals=iv, cand=cand)
        g = _score_lex(env, w, cs, ts, kernel)
        o = oracle.score_lex(p, iv, cand, cs, ts, n_threads=16)
        _assert_score_lex_equal(g, o, f"inst {inst}")


def test_stagewise_score_all_measured_and_no_candidate(env):
    """Every candidate revealed: scores 0, best -1, the stages from the
    certificate alone, on both scorers."""
    w = make_workload("tiny-2class-G16")
    p = w.problem
    iv = Intervals(w.intervals.cap_lo, w.intervals.cap_lo.copy(), w.intervals.tail_hi, w.intervals.tail_hi.copy(),
                   np.ones_like(w.intervals.measured))
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :8]), np.ascontiguousarray(w.tail_s[:, :, :8])
    note("stage-wise score, every candidate revealed")
    ww = SimpleNamespace(problem=p, intervals=iv, cand=w.cand)
    for kernel in (0, 1):
        g = _score_lex(env, ww, cs, ts, kernel)
        o = oracle.score_lex(p, iv, w.cand, cs, ts)
        _assert_score_lex_equal(g, o, f"all revealed, kernel {kernel}")
        assert np.all(g["score_maxmin"] == 0.0) and np.all(g["best"] == -1)


def test_stagewise_score_in_a_captured_graph(env):
    """fs_score_candidates_lex forks its certificate solves onto the
    context's second stream and joins them back with events, which stream
    capture follows: the call captured into a graph and replayed several
    times, with eager work and synchronizations between the replays, gives
    the eager call's outputs every time (the outputs are cleared before each
    replay)."""
    torch, fs, ctx = env
    w = make_workload("4class-G64", orders=[0, 1, 2])
    S = 16
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :S]), np.ascontiguousarray(w.tail_s[:, :, :S])
    div = fs.DeviceIntervals.from_host(w.intervals, "cuda:0")
    cand_d, cs_d, ts_d = _t(env, w.cand), _t(env, cs), _t(env, ts)
    note("stage-wise score captured in a graph, 4class-G64 orders 0-2 S=16")
    eager = fs.score_candidates_lex(ctx, w.problem, div, cand_d, cs_d, ts_d)
    torch.cuda.synchronize()
    want = {k: getattr(eager, k).clone() for k in ("score_maxmin", "score_goodput", "gap_maxmin", "gap_goodput",
                                                    "best")}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        plan = fs.ScoreLexPlan(ctx, w.problem, div, cand_d, cs_d, ts_d, stream=side)
        plan.run()
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            plan.run()
    torch.cuda.synchronize()
    for rep in range(4):
        for k in want:
            getattr(plan.out, k).fill_(-7)
        torch.cuda.synchronize()
        # eager work of the program between the replays
        other = fs.score_candidates(ctx, w.problem, div, cand_d, cs_d, ts_d)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in want:
            assert torch.equal(getattr(plan.out, k), want[k]), (rep, k)
        np.testing.assert_array_equal(other.score.cpu().numpy(), want["score_maxmin"].cpu().numpy())
