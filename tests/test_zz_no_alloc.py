"""fs_score_candidates_noalloc (the scorer for callers that cannot allocate:
its workspace is the library's static device scratch) against
fs_score_candidates on the same inputs, through the C ABI: scores, gaps,
best candidates and every tau of the dump bit for bit, on two calls in a
row, the second with a smaller input; sizes beyond the scratch are
rejected before any launch."""
import sys

import numpy as np
import pytest

from paper_2608_19659_amd.synth import make_workload

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


def _inputs(env, name, orders=None, S=None):
    torch, fs, ctx = env
    w = make_workload(name, orders=orders)
    S = S or w.n_samples
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")
    return (w, fs.DeviceIntervals.from_host(w.intervals, "cuda:0"), t(w.cand), t(w.cap_s[:, :, :S]),
            t(w.tail_s[:, :, :S]))


def _outputs(env, O, E, S, dump):
    torch, fs, ctx = env
    dev = "cuda:0"
    return fs.ScoreOutput(torch.full((O, E), -7.0, dtype=torch.float64, device=dev),
                          torch.full((O,), -7.0, dtype=torch.float64, device=dev),
                          torch.full((O,), -7, dtype=torch.int32, device=dev),
                          torch.full((O, E, S, 2), -7.0, device=dev) if dump else None)


def _compare(env, name, orders=None, S=None, dump=True):
    torch, fs, ctx = env
    w, iv, cand, cs, ts = _inputs(env, name, orders, S)
    O, E, S = cs.shape
    note(f"noalloc vs workspace scorer: {name} O={O} E={E} S={S} dump={dump}")
    ref = fs.score_candidates(ctx, w.problem, iv, cand, cs, ts, dump=dump)
    got = fs.score_candidates_noalloc(ctx, w.problem, iv, cand, cs, ts, _outputs(env, O, E, S, dump))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.score.cpu().numpy().view(np.uint64), ref.score.cpu().numpy().view(np.uint64))
    np.testing.assert_array_equal(got.gap_now.cpu().numpy().view(np.uint64), ref.gap_now.cpu().numpy().view(np.uint64))
    np.testing.assert_array_equal(got.best.cpu().numpy(), ref.best.cpu().numpy())
    if dump:
        np.testing.assert_array_equal(got.tau_dump.cpu().numpy().view(np.uint32),
                                      ref.tau_dump.cpu().numpy().view(np.uint32))


def test_two_calls_in_a_row_second_smaller(env):
    """The benchmark workload at full size, then a smaller one on the same
    scratch (whose first call left its contents behind)."""
    _compare(env, "4class-G64", dump=True)
    _compare(env, "paper-shaped-2class-G16", orders=[0, 3, 7], S=300, dump=True)
    _compare(env, "tiny-2class-G16", dump=False)


def test_other_kernels_use_the_scratch_too(env):
    torch, fs, ctx = env
    try:
        for kernel in (1, 2):
            ctx.set_score_kernel(kernel)
            _compare(env, "paper-shaped-2class-G16", orders=[1, 2], S=256, dump=True)
    finally:
        ctx.set_score_kernel(0)


def test_sizes_beyond_the_scratch_are_rejected(env):
    """65535 orders x 256 candidates x 4096 samples need more scratch than
    the library holds: FS_ERR_UNSUPPORTED from the host's size checks, which
    come before the array checks (every device pointer here is NULL, so
    nothing could be launched either way); sizes that fit pass the size
    check and stop at the NULL arrays instead."""
    torch, fs, ctx = env
    w = make_workload("4class-G64", orders=[0], with_samples=False)
    ref = fs._ProblemRef(w.problem)
    lib = fs.load_library()
    st = lib.fs_score_candidates_noalloc(ctx.handle, ref.ptr, fs._Intervals(), 65535, None, 256, None, None, 4096,
                                         None, None, None, None, None)
    assert st == fs.FS_ERR_UNSUPPORTED, lib.fs_last_error()
    assert b"scratch" in lib.fs_last_error()
    st = lib.fs_score_candidates_noalloc(ctx.handle, ref.ptr, fs._Intervals(), 16, None, 128, None, None, 4096,
                                         None, None, None, None, None)
    assert st == fs.FS_ERR_INVALID_ARGUMENT, lib.fs_last_error()
