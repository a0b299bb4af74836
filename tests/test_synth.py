"""Seeded input generator: determinism, shapes and the structure the
workloads are meant to have (interior knee, grid, samples inside intervals)."""
import hashlib

import numpy as np
import pytest

from paper_2608_19659_amd.synth import WORKLOADS, make_workload


def _digest(w):
    h = hashlib.sha256()
    for a in (w.problem.demand, w.problem.slo, w.intervals.cap_lo, w.intervals.cap_hi,
              w.intervals.tail_lo, w.intervals.tail_hi, w.intervals.measured, w.cand, w.cap_s, w.tail_s):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def test_deterministic():
    assert _digest(make_workload("tiny-2class-G16")) == _digest(make_workload("tiny-2class-G16"))
    assert _digest(make_workload("paper-shaped-2class-G16", orders=[3, 7])) == _digest(make_workload("paper-shaped-2class-G16", orders=[3, 7]))


def test_order_subset_matches_full_rows():
    full = make_workload("paper-shaped-2class-G16", orders=list(range(6)))
    sub = make_workload("paper-shaped-2class-G16", orders=[2, 5])
    for j, o in enumerate([2, 5]):
        np.testing.assert_array_equal(sub.intervals.cap_lo[j], full.intervals.cap_lo[o])
        np.testing.assert_array_equal(sub.intervals.measured[j], full.intervals.measured[o])
        np.testing.assert_array_equal(sub.cap_s[j], full.cap_s[o])
        np.testing.assert_array_equal(sub.tail_s[j], full.tail_s[o])


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_structure(name):
    c = WORKLOADS[name]
    w = make_workload(name, orders=[0, 1], with_samples=(c["G"] <= 64))
    p, iv = w.problem, w.intervals
    assert p.n_classes == c["K"] and p.budget == c["G"] and list(p.tp) == c["tp"]
    assert iv.cap_lo.shape == (2, p.n_cells)
    for a in (iv.cap_lo, iv.cap_hi):
        assert np.all(a * 64 == np.rint(a * 64)) and np.all(a >= 1 / 64)
    assert np.all(iv.cap_lo <= iv.cap_hi) and np.all(iv.tail_lo <= iv.tail_hi)
    m = iv.measured.astype(bool)
    assert np.all(iv.cap_lo[m] == iv.cap_hi[m]) and np.all(iv.tail_lo[m] == iv.tail_hi[m])
    # interior knee: per-GPU lower capacity of the initial intervals is largest
    # at TP4 in every (class, load); revealed cells hold the hidden truth instead
    k4 = list(p.tp).index(4)
    if c.get("structure"):
        # the truth has the refit's structure: per-GPU capacity unimodal over TP
        # with its knee at TP4, tail nondecreasing in the load; it lies inside
        for i in range(p.n_classes):
            for b in range(p.n_levels):
                per_gpu = np.array([w.truth_cap[p.cell(i, t, b)] / p.tp[t] for t in range(p.n_tp)])
                assert np.all(np.diff(per_gpu[:k4 + 1]) >= 0) and np.all(np.diff(per_gpu[k4:]) <= 0)
            for t in range(p.n_tp):
                assert np.all(np.diff([w.truth_tail[p.cell(i, t, b)] for b in range(p.n_levels)]) >= 0)
        assert np.all((iv.cap_lo <= w.truth_cap) & (w.truth_cap <= iv.cap_hi))
        assert np.all((iv.tail_lo <= w.truth_tail) & (w.truth_tail <= iv.tail_hi))
    else:
        for i in range(p.n_classes):
            for b in range(p.n_levels):
                if any(iv.measured[0][p.cell(i, t, b)] for t in range(p.n_tp)):
                    continue
                per_gpu = [iv.cap_lo[0][p.cell(i, t, b)] / p.tp[t] for t in range(p.n_tp)]
                assert all(per_gpu[k4] > v for t, v in enumerate(per_gpu) if t != k4)
    if w.cap_s is not None:
        lo = iv.cap_lo[:, w.cand][:, :, None]
        hi = iv.cap_hi[:, w.cand][:, :, None]
        assert np.all((w.cap_s >= lo) & (w.cap_s <= hi))
        assert np.all(w.cap_s * 64 == np.rint(w.cap_s * 64))
        lo = iv.tail_lo[:, w.cand][:, :, None]
        hi = iv.tail_hi[:, w.cand][:, :, None]
        assert np.all((w.tail_s >= lo) & (w.tail_s <= hi))


def test_interval_realisations_stay_inside():
    from paper_2608_19659_amd.synth import interval_realisations
    w = make_workload("4class-G64", with_samples=False)
    cap, tail = interval_realisations(w, 100)
    iv = w.intervals
    rows = np.arange(100) % iv.cap_lo.shape[0]
    assert (cap >= iv.cap_lo[rows]).all() and (cap <= iv.cap_hi[rows]).all()
    assert (tail >= iv.tail_lo[rows]).all() and (tail <= iv.tail_hi[rows]).all()
    assert np.array_equal(np.rint(cap * 64.0), cap * 64.0)
    c2, t2 = interval_realisations(w, 100)
    assert np.array_equal(cap, c2) and np.array_equal(tail, t2)
