"""Host-side checks of bench.py: the work model the roofline is computed
with (slots per scenario of the exclusion scorer, as the kernel runs it:
a scan for replica ranges of at most 4 counts, a crossing search beyond),
the algorithmic bytes of the benchmark workload, and the one-GPU limit."""
import math
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2608_19659_amd.synth import make_workload  # noqa: E402


def test_scan_slots():
    # per r: multiply + quotient (3) + a (max,min) step into each
    # realisation (2 x 1.5); per scenario 7
    assert bench.excl_slots_per_scenario(1) == 14
    assert bench.excl_slots_per_scenario(2) == 21
    assert bench.excl_slots_per_scenario(4) == 35


def test_search_slots():
    # per realisation ceil(log2(n + 1)) compare+select steps, multiply +
    # quotient (4), the max of two candidates into the accumulator (2)
    for n, steps in [(5, 3), (7, 3), (8, 4), (31, 5), (32, 6), (63, 6), (64, 7), (1006, 10)]:
        assert math.ceil(math.log2(n + 1)) == steps
        assert bench.excl_slots_per_scenario(n) == 2 * (2 * steps + 6) + 7


def test_benchmark_workload_work():
    w = make_workload("4class-G64")
    O, E, S = w.cap_s.shape
    measured = w.intervals.measured[:, w.cand].astype(bool)
    live = [(o, e) for o in range(O) for e in range(E) if not measured[o, e]]
    slots, nbytes, mean_ne, sampled = bench.excl_work(w.problem, w.cand, live, S)
    assert sampled == 3_649_536 and nbytes == 8 * sampled
    assert abs(slots - 93_114_368) < 1
    assert mean_ne == 3.75
    # the binding roofline of this workload is HBM
    assert nbytes / bench.HBM_PEAK_BYTES > slots / bench.VALU_PEAK_OPS


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
