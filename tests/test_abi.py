"""The C ABI library loads, exports every entry point include/fleetsieve.h
declares, and rejects malformed problems on the host (no GPU needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT
from paper_2608_19659_amd import fleetsieve as fs
from paper_2608_19659_amd.synth import Problem

HEADER = os.path.join(ROOT, "include", "fleetsieve.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fs.LIB_PATH):
        from paper_2608_19659_amd.build import build_library
        build_library()
    return fs.load_library()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(fs_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_surface():
    assert set(_declared()) == set(fs.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in _declared():
        assert hasattr(lib, name), name


def _problem(**kw):
    base = dict(tp=[1, 2, 4, 8], levels=[0.5, 1.0, 2.0], demand=[4.0, 2.0], slo=[30.0, 30.0], budget=16)
    base.update(kw)
    return Problem(**base)


def _status(problem):
    ref = fs._ProblemRef(problem)
    return fs.load_library().fs_validate_problem(ref.ptr)


def test_valid_problem(lib):
    assert _status(_problem()) == fs.FS_OK
    assert fs.workspace_size(_problem()) > 0


@pytest.mark.parametrize("bad", [
    dict(tp=[2, 1, 4, 8]),                 # not ascending
    dict(tp=[0, 2, 4, 8]),                 # TP < 1
    dict(tp=[1, 2, 2, 8]),                 # duplicate
    dict(budget=0),
    dict(budget=4097),
    dict(tp=[2, 4], budget=1),             # below the smallest TP
    dict(levels=[0.5, 0.5, 2.0]),
    dict(levels=[0.0, 1.0, 2.0]),
    dict(levels=[0.5, 1.0, np.inf]),
    dict(demand=[0.0, 2.0]),
    dict(demand=[np.nan, 2.0]),
    dict(demand=[2.0**33, 2.0]),
    dict(slo=[np.nan, 30.0]),
    dict(floor_rps=[-1.0, 0.0]),
    dict(floor_rps=[np.inf, 0.0]),
], ids=lambda d: ",".join(f"{k}={v}" for k, v in d.items()))
def test_invalid_problems_rejected(lib, bad):
    assert _status(_problem(**bad)) == fs.FS_ERR_INVALID_ARGUMENT
    assert fs.load_library().fs_last_error()


def test_too_many_classes(lib):
    K = 65
    p = _problem(demand=np.ones(K), slo=np.full(K, 30.0))
    assert _status(p) == fs.FS_ERR_INVALID_ARGUMENT


def test_null_problem_and_sizes(lib):
    out = ctypes.c_size_t()
    assert lib.fs_validate_problem(None) == fs.FS_ERR_INVALID_ARGUMENT
    ref = fs._ProblemRef(_problem())
    assert lib.fs_workspace_size(ref.ptr, -1, 0, 0, ctypes.byref(out)) == fs.FS_ERR_INVALID_ARGUMENT
    assert lib.fs_workspace_size(ref.ptr, 0, 0, 0, None) == fs.FS_ERR_INVALID_ARGUMENT


def test_workspace_grows_with_work(lib):
    p = _problem()
    small = fs.workspace_size(p, 1, 8, 64)
    big = fs.workspace_size(p, 200, 48, 1024)
    assert big > small > 0


def test_null_context_is_rejected_before_any_device_call(lib):
    ref = fs._ProblemRef(_problem())
    st = lib.fs_solve_batch(None, ref.ptr, None, None, 0, fs._Alloc(), None, 0, None)
    assert st == fs.FS_ERR_INVALID_ARGUMENT
    st = lib.fs_score_candidates(None, ref.ptr, fs._Intervals(), 0, None, 0, None, None, 0, None, None,
                                 None, None, None, 0, None)
    assert st == fs.FS_ERR_INVALID_ARGUMENT
    st = lib.fs_certify(None, ref.ptr, fs._Intervals(), 0, 0.05, None, fs._Alloc(), fs._Alloc(), None,
                        None, 0, None)
    assert st == fs.FS_ERR_INVALID_ARGUMENT
    assert lib.fs_context_set_option(None, fs.OPT_SCORE_KERNEL, 0) == fs.FS_ERR_INVALID_ARGUMENT


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(fs, "_lib", None)
    monkeypatch.setattr(fs, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(fs.FleetSieveError):
        fs.load_library()
