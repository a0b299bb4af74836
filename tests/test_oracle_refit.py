"""Pins of the interval refit (Algorithm 1's fit step; Section 4.1's
interior-knee structural prior with measured cells): a hand-derived case
(tests/golden/refit.json), the closed form of the capacity bound, and
invariants -- it never widens an interval, leaves measured cells alone, is
idempotent, and keeps any truth that satisfies the prior."""
from types import SimpleNamespace

import numpy as np
import pytest

import oracle
from conftest import load_golden
from paper_2608_19659_amd.synth import Problem, make_workload


def _iv(d, O=1):
    return SimpleNamespace(**{k: np.array(v, np.uint8 if k == "measured" else np.float32).reshape(O, -1)
                              for k, v in d.items()})


def test_hand_derived_case():
    g = load_golden("refit.json")
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"])
    f = oracle.refit_intervals(p, _iv(g["before"]))
    for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi"):
        assert list(getattr(f, k)[0]) == g["after"][k], k
    assert list(f.measured[0]) == g["before"]["measured"]


def _random_state(name, seed, frac):
    w = make_workload(name, orders=list(range(4)), with_samples=False)
    rng = np.random.default_rng(seed)
    iv = w.intervals
    ms = (rng.random(iv.measured.shape) < frac).astype(np.uint8) | iv.measured
    cl, ch = iv.cap_lo.copy(), iv.cap_hi.copy()
    tl, th = iv.tail_lo.copy(), iv.tail_hi.copy()
    for o in range(ms.shape[0]):
        m = ms[o].astype(bool)
        cl[o, m] = ch[o, m] = w.truth_cap[m]
        tl[o, m] = th[o, m] = w.truth_tail[m]
    return w, SimpleNamespace(cap_lo=cl, cap_hi=ch, tail_lo=tl, tail_hi=th, measured=ms)


@pytest.mark.parametrize("name", ["paper-shaped-2class-G16-knee", "4class-G64-knee"])
@pytest.mark.parametrize("seed", range(4))
def test_truth_with_the_structure_stays_inside(name, seed):
    w, iv = _random_state(name, seed, 0.3)
    f = oracle.refit_intervals(w.problem, iv)
    assert np.all((f.cap_lo <= w.truth_cap) & (w.truth_cap <= f.cap_hi))
    assert np.all((f.tail_lo <= w.truth_tail) & (w.truth_tail <= f.tail_hi))
    assert (f.cap_lo > iv.cap_lo).any() and ((f.tail_lo > iv.tail_lo) | (f.tail_hi < iv.tail_hi)).any()


@pytest.mark.parametrize("name", ["paper-shaped-2class-G16", "4class-G64", "16class-G1024"])
def test_invariants_without_the_structure(name):
    """On tables that need not satisfy the prior: never wider, measured
    cells untouched, nonempty, idempotent; the capacity bound equals
    t * min(best per-GPU value measured below t, best measured above t)."""
    w, iv = _random_state(name, 7, 0.4)
    p = w.problem
    f = oracle.refit_intervals(p, iv)
    m = iv.measured.astype(bool)
    assert np.all(f.cap_lo >= iv.cap_lo) and np.array_equal(f.cap_hi, iv.cap_hi)
    assert np.all(f.tail_lo >= iv.tail_lo) and np.all(f.tail_hi <= iv.tail_hi)
    assert np.all(f.cap_lo <= f.cap_hi) and np.all(f.tail_lo <= f.tail_hi)
    for k in ("cap_lo", "tail_lo", "tail_hi"):
        assert np.array_equal(getattr(f, k)[m], getattr(iv, k)[m])
    g = oracle.refit_intervals(p, f)
    for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi"):
        assert np.array_equal(getattr(g, k), getattr(f, k)), k
    T, B = p.n_tp, p.n_levels
    tp = np.asarray(p.tp, np.float64)
    for o in range(iv.cap_lo.shape[0]):
        for i in range(p.n_classes):
            for b in range(B):
                cells = [p.cell(i, t, b) for t in range(T)]
                per = np.array([iv.cap_lo[o, c] / tp[t] if m[o, c] else -np.inf for t, c in enumerate(cells)])
                for t, c in enumerate(cells):
                    if m[o, c]:
                        continue
                    left, right = per[:t].max(initial=-np.inf), per[t + 1:].max(initial=-np.inf)
                    bound = tp[t] * min(left, right)
                    want = iv.cap_lo[o, c]
                    if np.isfinite(bound):
                        v = np.float32(bound)
                        v = v if float(v) <= bound else np.nextafter(v, np.float32(-np.inf))
                        want = max(want, v)
                    expect = want if want <= iv.cap_hi[o, c] else iv.cap_lo[o, c]
                    assert f.cap_lo[o, c] == expect, (o, i, b, t)


def test_round_down_of_the_capacity_bound():
    """A per-GPU bound that binary32 cannot hold is rounded down, so the
    refitted lower bound never exceeds the true value at the bound."""
    p = Problem(tp=[1, 3, 9], levels=[1.0], demand=[1.0], slo=[30.0], budget=9)
    iv = _iv({"cap_lo": [1.0, 0.1, 1.0], "cap_hi": [1.0, 5.0, 1.0], "tail_lo": [1.0] * 3, "tail_hi": [1.0] * 3,
              "measured": [1, 0, 1]})
    f = oracle.refit_intervals(p, iv)
    exact = 3.0 * (1.0 / 9.0)  # 1/3, not a binary32 value
    assert float(f.cap_lo[0, 1]) <= exact < float(np.nextafter(f.cap_lo[0, 1], np.float32(1)))


def test_loop_with_refit_on_structured_tables():
    """The loop with the fit step certifies with zero regret on a table
    that satisfies the prior, and never needs more reveals than without it
    on these orders."""
    w = make_workload("4class-G64-knee", orders=list(range(6)))
    O = len(w.orders)
    tc = np.repeat(w.truth_cap[None], O, axis=0)
    tt = np.repeat(w.truth_tail[None], O, axis=0)
    cs, ts = np.ascontiguousarray(w.cap_s[:, :, :32]), np.ascontiguousarray(w.tail_s[:, :, :32])
    a = oracle.profile_loop(w.problem, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, n_threads=8, refit=True)
    b = oracle.profile_loop(w.problem, w.intervals, tc, tt, w.cand, cs, ts, eps=0.05, n_threads=8)
    assert (a.state == 1).all() and (a.regret == 0).all()
    assert a.gpu_seconds.sum() <= b.gpu_seconds.sum()


def test_clamp_into_refitted_intervals_hand_derived():
    """Samples are clamped into the refitted intervals (Algorithm 1 refits
    before every score): below a raised cap_lo, above a lowered tail_hi, and
    exactly at a bound (tests/golden/clamp_samples.json)."""
    g = load_golden("clamp_samples.json")
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"])
    iv = _iv(g["intervals"])
    f = oracle.refit_intervals(p, iv)
    for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi"):
        assert list(getattr(f, k)[0]) == g["refit"][k], k
    cs, ts = np.array([g["cap_s"]], np.float32), np.array([g["tail_s"]], np.float32)
    c2, t2 = oracle.clamp_samples(f, g["cand"], cs, ts)
    assert c2.tolist() == [g["clamped_cap_s"]] and t2.tolist() == [g["clamped_tail_s"]]
    # the pin separates the refitted intervals from the initial ones
    c0, t0 = oracle.clamp_samples(iv, g["cand"], cs, ts)
    assert c0.tolist() != [g["clamped_cap_s"]] and t0.tolist() != [g["clamped_tail_s"]]


def test_clamp_properties():
    """On a workload: clamped samples lie inside the intervals, samples
    already inside are unchanged, and clamping is idempotent."""
    w, iv = _random_state("4class-G64-knee", 3, 0.3)
    w = make_workload("4class-G64-knee", orders=list(range(4)))
    f = oracle.refit_intervals(w.problem, iv)
    cs, ts = oracle.clamp_samples(f, w.cand, w.cap_s[:, :, :256], w.tail_s[:, :, :256])
    lo, hi = f.cap_lo[:, w.cand][:, :, None], f.cap_hi[:, w.cand][:, :, None]
    assert np.all((cs >= lo) & (cs <= hi))
    tl, th = f.tail_lo[:, w.cand][:, :, None], f.tail_hi[:, w.cand][:, :, None]
    assert np.all((ts >= tl) & (ts <= th))
    inside = (w.cap_s[:, :, :256] >= lo) & (w.cap_s[:, :, :256] <= hi)
    assert np.array_equal(cs[inside], w.cap_s[:, :, :256][inside])
    c2, t2 = oracle.clamp_samples(f, w.cand, cs, ts)
    assert np.array_equal(c2, cs) and np.array_equal(t2, ts)
    assert (cs != w.cap_s[:, :, :256]).any()  # the refit moved some samples


@pytest.mark.parametrize("case", range(2))
def test_fit_step_saves_a_reveal_hand_derived(case):
    """A loop in which the fit step decides (tests/golden/refit_loop.json):
    the refitted tail of the only candidate lies above the SLO, the gap
    closes and the loop certifies with no reveal, where the loop without
    the fit step pays one reveal (300 GPU-s) for the same allocation."""
    from paper_2608_19659_amd.synth import Intervals
    g = load_golden("refit_loop.json")
    c = g["cases"][case]
    p = Problem(tp=g["tp"], levels=g["levels"], demand=g["demand"], slo=g["slo"], budget=g["budget"])
    d = g["intervals"]
    iv = Intervals(*(np.array([d[k]], np.float32) for k in ("cap_lo", "cap_hi", "tail_lo", "tail_hi")),
                   np.array([d["measured"]], np.uint8))
    r = oracle.profile_loop(p, iv, [g["truth_cap"]], [g["truth_tail"]], g["cand"], np.array([g["cap_s"]], np.float32),
                            np.array([g["tail_s"]], np.float32), eps=g["eps"], refit=c["refit"])
    assert r.state[0] == oracle.CERTIFIED_FEASIBLE
    assert r.rounds[0] == c["rounds"] and list(r.reveals[0][: r.rounds[0]]) == c["reveals"]
    assert r.gpu_seconds[0] == c["gpu_seconds"]
    assert r.final[0].tp_index == c["final_tp_index"] and r.final[0].replicas == c["final_replicas"]
    assert r.final[0].tau == np.float32(c["final_tau"])
    assert r.tau_truth[0] == np.float32(c["tau_truth"]) and r.tau_oracle[0] == np.float32(c["tau_oracle"])
