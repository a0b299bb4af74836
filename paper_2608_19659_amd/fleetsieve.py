"""Thin ctypes binding of libfleetsieve (C ABI in include/fleetsieve.h).

Argument marshalling only: every step runs in the HIP library.  Device
arrays are torch tensors on a ROCm device (torch supplies memory and the
current stream); the problem statement is host data.  There is no fallback:
if ``libfleetsieve.so`` is missing or the device is not gfx950 the calls
raise.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# FLEETSIEVE_LIB selects another build of the library (for example one whose
# host code is compiled with sanitizers); the default is the in-tree build.
LIB_PATH = os.environ.get("FLEETSIEVE_LIB") or os.path.join(_HERE, "libfleetsieve.so")

FS_OK, FS_ERR_INVALID_ARGUMENT, FS_ERR_UNSUPPORTED, FS_ERR_WORKSPACE_TOO_SMALL, FS_ERR_DEVICE, \
    FS_ERR_INTERNAL = range(6)
UNDECIDED, CERTIFIED_FEASIBLE, CERTIFIED_INFEASIBLE = 0, 1, 2
TP_NONE = 0xFF
OPT_SCORE_KERNEL = 1
OPT_KERNEL_TIMING = 2
OPT_SAMPLES_PER_LANE = 3
OPT_SCORER_WAVES = 5
OPT_SETUP = 6
OPT_LOOP_OBJECTIVE = 7
OPT_LOOP_REFIT = 8
OPT_THRESHOLD_SEARCH = 9
OBJECTIVE_MAXMIN, OBJECTIVE_LEXICOGRAPHIC = 0, 1
KERNEL_AUTO, KERNEL_WAVE, KERNEL_LANE, KERNEL_EXCLUSION = 0, 1, 2, 3

EXPORTED = ("fs_context_create", "fs_context_destroy", "fs_context_set_option", "fs_context_kernel_timing",
            "fs_last_error",
            "fs_validate_problem", "fs_workspace_size", "fs_solve_batch", "fs_score_candidates",
            "fs_certify", "fs_loop_workspace_size", "fs_profile_loop", "fs_reduce_cells", "fs_reduce_samples",
            "fs_solve_batch_lex", "fs_certify_lex", "fs_refit_intervals", "fs_loop_refit_workspace_size",
            "fs_score_lex_workspace_size", "fs_score_candidates_lex", "fs_clamp_samples",
            "fs_score_candidates_noalloc")
POLICY_SCORE, POLICY_ORDER = 0, 1
CELL_SECONDS = 300.0


class FleetSieveError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libfleetsieve status {status}: {message}")
        self.status = status


class _Problem(ctypes.Structure):
    _fields_ = [("n_classes", ctypes.c_int32), ("n_tp", ctypes.c_int32),
                ("n_levels", ctypes.c_int32), ("budget", ctypes.c_int32),
                ("tp", ctypes.c_void_p), ("levels", ctypes.c_void_p),
                ("demand", ctypes.c_void_p), ("slo", ctypes.c_void_p),
                ("floor_rps", ctypes.c_void_p)]


class _Intervals(ctypes.Structure):
    _fields_ = [("cap_lo", ctypes.c_void_p), ("cap_hi", ctypes.c_void_p),
                ("tail_lo", ctypes.c_void_p), ("tail_hi", ctypes.c_void_p),
                ("measured", ctypes.c_void_p)]


class _Alloc(ctypes.Structure):
    _fields_ = [("objective", ctypes.c_void_p), ("tp_index", ctypes.c_void_p),
                ("replicas", ctypes.c_void_p), ("floors_met", ctypes.c_void_p),
                ("goodput", ctypes.c_void_p)]


class _SloPolicy(ctypes.Structure):
    _fields_ = [("n_metrics", ctypes.c_int32), ("limit", ctypes.c_void_p), ("success_min", ctypes.c_void_p)]


class _LoopOut(ctypes.Structure):
    _fields_ = [("state", ctypes.c_void_p), ("finished", ctypes.c_void_p), ("rounds", ctypes.c_void_p),
                ("gpu_seconds", ctypes.c_void_p), ("reveals", ctypes.c_void_p), ("final_alloc", _Alloc),
                ("tau_truth", ctypes.c_void_p), ("tau_oracle", ctypes.c_void_p)]


_lib = None


def load_library():
    """Load libfleetsieve.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise FleetSieveError(FS_ERR_INTERNAL, f"{LIB_PATH} is not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    P = ctypes.POINTER(_Problem)
    lib.fs_context_create.argtypes = [ctypes.c_int, ctypes.POINTER(vp)]
    lib.fs_context_destroy.argtypes = [vp]
    lib.fs_context_destroy.restype = None
    lib.fs_context_set_option.argtypes = [vp, ctypes.c_int, i64]
    lib.fs_context_kernel_timing.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)]
    lib.fs_last_error.restype = ctypes.c_char_p
    lib.fs_validate_problem.argtypes = [P]
    lib.fs_workspace_size.argtypes = [P, i32, i32, i32, ctypes.POINTER(sz)]
    lib.fs_solve_batch.argtypes = [vp, P, vp, vp, i64, _Alloc, vp, sz, vp]
    lib.fs_score_candidates.argtypes = [vp, P, _Intervals, i32, vp, i32, vp, vp, i32, vp, vp, vp, vp,
                                        vp, sz, vp]
    lib.fs_certify.argtypes = [vp, P, _Intervals, i32, ctypes.c_float, vp, _Alloc, _Alloc, vp, vp, sz, vp]
    lib.fs_loop_workspace_size.argtypes = [P, i32, i32, i32, ctypes.POINTER(sz)]
    lib.fs_profile_loop.argtypes = [vp, P, _Intervals, i32, vp, vp, vp, i32, vp, vp, i32, ctypes.c_float,
                                    ctypes.c_int, vp, i32, i32, _LoopOut, vp, sz, vp]
    lib.fs_score_lex_workspace_size.argtypes = [P, i32, i32, i32, ctypes.POINTER(sz)]
    lib.fs_score_candidates_lex.argtypes = [vp, P, _Intervals, i32, vp, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp,
                                            sz, vp]
    lib.fs_refit_intervals.argtypes = [vp, P, _Intervals, i32, vp, vp, vp, vp]
    lib.fs_loop_refit_workspace_size.argtypes = [P, i32, i32, i32, ctypes.POINTER(sz)]
    lib.fs_clamp_samples.argtypes = [vp, P, _Intervals, i32, vp, i32, vp, vp, i32, vp, vp, vp]
    lib.fs_score_candidates_noalloc.argtypes = [vp, P, _Intervals, i32, vp, i32, vp, vp, i32, vp, vp, vp, vp, vp]
    lib.fs_solve_batch_lex.argtypes = [vp, P, vp, vp, i64, _Alloc, vp, vp, sz, vp]
    lib.fs_certify_lex.argtypes = [vp, P, _Intervals, i32, ctypes.c_float, vp, _Alloc, _Alloc, vp, vp, vp, sz, vp]
    Q = ctypes.POINTER(_SloPolicy)
    lib.fs_reduce_cells.argtypes = [vp, P, Q, vp, vp, i64, vp, vp]
    lib.fs_reduce_samples.argtypes = [vp, P, Q, vp, i32, vp, vp, i32, i32, vp, vp]
    for name in EXPORTED:
        if name != "fs_context_destroy":
            getattr(lib, name).restype = ctypes.c_int
    lib.fs_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int):
    if status != FS_OK:
        msg = load_library().fs_last_error()
        raise FleetSieveError(status, msg.decode() if msg else "")


class _ProblemRef:
    """Host copy of a problem statement kept alive for the duration of a call."""

    def __init__(self, problem):
        self.tp = np.ascontiguousarray(problem.tp, dtype=np.int32)
        self.levels = np.ascontiguousarray(problem.levels, dtype=np.float32)
        self.demand = np.ascontiguousarray(problem.demand, dtype=np.float32)
        self.slo = np.ascontiguousarray(problem.slo, dtype=np.float32)
        fl = getattr(problem, "floor_rps", None)
        self.floor = None if fl is None else np.ascontiguousarray(fl, dtype=np.float32)
        self.K, self.NT, self.B = len(self.demand), len(self.tp), len(self.levels)
        self.N = self.K * self.NT * self.B
        self.s = _Problem(self.K, self.NT, self.B, int(problem.budget),
                          self.tp.ctypes.data, self.levels.ctypes.data, self.demand.ctypes.data,
                          self.slo.ctypes.data, None if self.floor is None else self.floor.ctypes.data)

    @property
    def ptr(self):
        return ctypes.byref(self.s)


def _torch():
    import torch
    return torch


def _dev_ptr(t, dtype, shape=None, name="array"):
    torch = _torch()
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise FleetSieveError(FS_ERR_INVALID_ARGUMENT, f"{name} must be a torch tensor on a ROCm device")
    if t.dtype != dtype:
        raise FleetSieveError(FS_ERR_INVALID_ARGUMENT, f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise FleetSieveError(FS_ERR_INVALID_ARGUMENT, f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise FleetSieveError(FS_ERR_INVALID_ARGUMENT, f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr()


def _stream(device, stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


class Context:
    """A libfleetsieve context on one HIP device."""

    def __init__(self, device: int = 0):
        lib = load_library()
        h = ctypes.c_void_p()
        _check(lib.fs_context_create(int(device), ctypes.byref(h)))
        self.handle = h
        self.device = int(device)
        self._ws = None

    def set_option(self, option: int, value: int):
        _check(load_library().fs_context_set_option(self.handle, int(option), int(value)))

    def set_score_kernel(self, kernel: int):
        self.set_option(OPT_SCORE_KERNEL, kernel)

    def kernel_timing(self):
        """(total milliseconds, launches) of the scoring kernel since the
        last query; needs set_option(OPT_KERNEL_TIMING, n), which launches
        it n times back to back between each pair of events."""
        ms, n = ctypes.c_double(), ctypes.c_int64()
        _check(load_library().fs_context_kernel_timing(self.handle, ctypes.byref(ms), ctypes.byref(n)))
        return float(ms.value), int(n.value)

    def close(self):
        if self.handle:
            load_library().fs_context_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace(self, nbytes: int):
        """A device workspace of at least nbytes, reused across calls that
        run on the same stream."""
        torch = _torch()
        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=f"cuda:{self.device}")
        return self._ws


def validate_problem(problem):
    ref = _ProblemRef(problem)
    _check(load_library().fs_validate_problem(ref.ptr))


def workspace_size(problem, n_orders: int = 0, n_cand: int = 0, n_samples: int = 0) -> int:
    ref = _ProblemRef(problem)
    out = ctypes.c_size_t()
    _check(load_library().fs_workspace_size(ref.ptr, int(n_orders), int(n_cand), int(n_samples),
                                            ctypes.byref(out)))
    return int(out.value)


def _alloc_tensors(n, K, device):
    torch = _torch()
    return dict(objective=torch.empty(n, dtype=torch.float32, device=device),
                tp_index=torch.empty((n, K), dtype=torch.uint8, device=device),
                replicas=torch.empty((n, K), dtype=torch.int16, device=device),
                floors_met=torch.empty(n, dtype=torch.uint8, device=device),
                goodput=torch.empty(n, dtype=torch.float32, device=device))


def _alloc_struct(d):
    return _Alloc(d["objective"].data_ptr(), d["tp_index"].data_ptr(), d["replicas"].data_ptr(),
                  d["floors_met"].data_ptr(), d["goodput"].data_ptr())


def solve_batch(ctx: Context, problem, cap, tail, stream=None, workspace=None):
    """Dense batch solve; cap, tail are float32 [n, N] device tensors.
    Returns a dict of device tensors (objective, tp_index, replicas,
    floors_met, goodput); replicas are uint16 values stored as int16."""
    torch = _torch()
    ref = _ProblemRef(problem)
    n = int(cap.shape[0]) if cap.dim() == 2 else 0
    pc = _dev_ptr(cap, torch.float32, (n, ref.N), "cap")
    pt = _dev_ptr(tail, torch.float32, (n, ref.N), "tail")
    out = _alloc_tensors(n, ref.K, cap.device)
    ws_bytes = workspace_size(problem)
    ws = workspace if workspace is not None else ctx.workspace(ws_bytes)
    _check(load_library().fs_solve_batch(ctx.handle, ref.ptr, pc, pt, n, _alloc_struct(out), ws.data_ptr(),
                                         ws.numel(), _stream(cap.device, stream)))
    return out


def solve_batch_lex(ctx: Context, problem, cap, tail, stream=None, workspace=None):
    """Dense batch solve under the whole lexicographic objective (levels
    1-4, fs_solve_batch_lex).  As solve_batch, plus goodput64: level (3)'s
    binary64 total per scenario."""
    torch = _torch()
    ref = _ProblemRef(problem)
    n = int(cap.shape[0]) if cap.dim() == 2 else 0
    pc = _dev_ptr(cap, torch.float32, (n, ref.N), "cap")
    pt = _dev_ptr(tail, torch.float32, (n, ref.N), "tail")
    out = _alloc_tensors(n, ref.K, cap.device)
    out["goodput64"] = torch.empty(n, dtype=torch.float64, device=cap.device)
    ws_bytes = workspace_size(problem)
    ws = workspace if workspace is not None else ctx.workspace(ws_bytes)
    _check(load_library().fs_solve_batch_lex(ctx.handle, ref.ptr, pc, pt, n, _alloc_struct(out),
                                             out["goodput64"].data_ptr(), ws.data_ptr(), ws.numel(),
                                             _stream(cap.device, stream)))
    return out


@dataclass
class DeviceIntervals:
    cap_lo: object
    cap_hi: object
    tail_lo: object
    tail_hi: object
    measured: object

    @staticmethod
    def from_host(iv, device):
        torch = _torch()
        return DeviceIntervals(*(torch.from_numpy(np.ascontiguousarray(a)).to(device)
                                 for a in (iv.cap_lo, iv.cap_hi, iv.tail_lo, iv.tail_hi, iv.measured)))


def _intervals_struct(iv, O, N):
    torch = _torch()
    return _Intervals(_dev_ptr(iv.cap_lo, torch.float32, (O, N), "cap_lo"),
                      _dev_ptr(iv.cap_hi, torch.float32, (O, N), "cap_hi"),
                      _dev_ptr(iv.tail_lo, torch.float32, (O, N), "tail_lo"),
                      _dev_ptr(iv.tail_hi, torch.float32, (O, N), "tail_hi"),
                      _dev_ptr(iv.measured, torch.uint8, (O, N), "measured"))


@dataclass
class ScoreOutput:
    score: object     # [O, E] float64
    gap_now: object   # [O] float64
    best: object      # [O] int32
    tau_dump: object  # [O, E, S, 2] float32 or None


class ScorePlan:
    """One fs_score_candidates call with its arguments checked and
    marshalled once.  run() enqueues the call again on the same device
    buffers (whose contents may change between runs); every run executes the
    whole scoring path on the GPU.  iv holds [O, N] device tensors, cand an
    int32 [E] device tensor, cap_s / tail_s float32 [O, E, S] device tensors."""

    def __init__(self, ctx: Context, problem, iv: DeviceIntervals, cand, cap_s, tail_s, dump: bool = False,
                 stream=None, workspace=None, out: ScoreOutput | None = None):
        torch = _torch()
        self._ref = _ProblemRef(problem)
        O = int(iv.cap_lo.shape[0])
        E = int(cand.shape[0])
        S = int(cap_s.shape[2]) if E > 0 else 0
        dev = iv.cap_lo.device
        self._ivs = _intervals_struct(iv, O, self._ref.N)
        pcand = _dev_ptr(cand, torch.int32, (E,), "cand")
        pcs = _dev_ptr(cap_s, torch.float32, (O, E, S), "cap_s")
        pts = _dev_ptr(tail_s, torch.float32, (O, E, S), "tail_s")
        if out is None:
            out = ScoreOutput(torch.empty((O, E), dtype=torch.float64, device=dev),
                              torch.empty(O, dtype=torch.float64, device=dev),
                              torch.empty(O, dtype=torch.int32, device=dev),
                              torch.empty((O, E, S, 2), dtype=torch.float32, device=dev) if dump else None)
        ws_bytes = workspace_size(problem, O, E, S)
        ws = workspace if workspace is not None else ctx.workspace(ws_bytes)
        self.out, self._ws, self._keep = out, ws, (iv, cand, cap_s, tail_s)
        self._fn = load_library().fs_score_candidates
        self._args = (ctx.handle, self._ref.ptr, self._ivs, O, pcand, E, pcs, pts, S,
                      _dev_ptr(out.score, torch.float64, (O, E), "score"),
                      _dev_ptr(out.gap_now, torch.float64, (O,), "gap_now"),
                      _dev_ptr(out.best, torch.int32, (O,), "best"),
                      _dev_ptr(out.tau_dump, torch.float32, (O, E, S, 2), "tau_dump"),
                      ws.data_ptr(), ws.numel(), _stream(dev, stream))

    def run(self) -> ScoreOutput:
        _check(self._fn(*self._args))
        return self.out


NOALLOC_SCRATCH_BYTES = 32 << 20


def score_candidates_noalloc(ctx: Context, problem, iv: DeviceIntervals, cand, cap_s, tail_s,
                             out: "ScoreOutput", stream=None) -> "ScoreOutput":
    """fs_score_candidates_noalloc: the scorer without a workspace (the
    library's static device scratch); the caller passes the outputs."""
    torch = _torch()
    ref = _ProblemRef(problem)
    O = int(iv.cap_lo.shape[0])
    E = int(cand.shape[0])
    S = int(cap_s.shape[2]) if E > 0 else 0
    ivs = _intervals_struct(iv, O, ref.N)
    _check(load_library().fs_score_candidates_noalloc(
        ctx.handle, ref.ptr, ivs, O, _dev_ptr(cand, torch.int32, (E,), "cand"),
        E, _dev_ptr(cap_s, torch.float32, (O, E, S), "cap_s"), _dev_ptr(tail_s, torch.float32, (O, E, S), "tail_s"),
        S, _dev_ptr(out.score, torch.float64, (O, E), "score"), _dev_ptr(out.gap_now, torch.float64, (O,), "gap_now"),
        _dev_ptr(out.best, torch.int32, (O,), "best"), _dev_ptr(out.tau_dump, torch.float32, (O, E, S, 2), "tau_dump"),
        _stream(iv.cap_lo.device, stream)))
    return out


def score_candidates(ctx: Context, problem, iv: DeviceIntervals, cand, cap_s, tail_s, dump: bool = False,
                     stream=None, workspace=None, out: ScoreOutput | None = None) -> ScoreOutput:
    """Acquisition scores (fs_score_candidates), one call."""
    return ScorePlan(ctx, problem, iv, cand, cap_s, tail_s, dump, stream, workspace, out).run()


@dataclass
class CertifyOutput:
    state: object
    gap: object
    cons: dict
    opt: dict


def certify(ctx: Context, problem, iv: DeviceIntervals, eps: float = 0.05, stream=None,
            workspace=None) -> CertifyOutput:
    torch = _torch()
    ref = _ProblemRef(problem)
    O = int(iv.cap_lo.shape[0])
    dev = iv.cap_lo.device
    ivs = _intervals_struct(iv, O, ref.N)
    state = torch.empty(O, dtype=torch.int32, device=dev)
    gap = torch.empty(O, dtype=torch.float64, device=dev)
    cons = _alloc_tensors(O, ref.K, dev)
    opt = _alloc_tensors(O, ref.K, dev)
    ws_bytes = workspace_size(problem)
    ws = workspace if workspace is not None else ctx.workspace(ws_bytes)
    _check(load_library().fs_certify(ctx.handle, ref.ptr, ivs, O, float(eps), state.data_ptr(),
                                     _alloc_struct(cons), _alloc_struct(opt), gap.data_ptr(), ws.data_ptr(),
                                     ws.numel(), _stream(dev, stream)))
    return CertifyOutput(state, gap, cons, opt)


@dataclass
class CertifyLexOutput:
    state: object
    gap_maxmin: object   # [O] float64, tau+ - tau-
    gap_goodput: object  # [O] float64, |gp+ - gp-| / max(gp+, gp-)
    cons: dict
    opt: dict


def certify_lex(ctx: Context, problem, iv: DeviceIntervals, eps: float = 0.05, stream=None,
                workspace=None) -> CertifyLexOutput:
    """Certificate with the stage-wise gap under the whole objective
    (fs_certify_lex)."""
    torch = _torch()
    ref = _ProblemRef(problem)
    O = int(iv.cap_lo.shape[0])
    dev = iv.cap_lo.device
    ivs = _intervals_struct(iv, O, ref.N)
    state = torch.empty(O, dtype=torch.int32, device=dev)
    gmm = torch.empty(O, dtype=torch.float64, device=dev)
    ggp = torch.empty(O, dtype=torch.float64, device=dev)
    cons = _alloc_tensors(O, ref.K, dev)
    opt = _alloc_tensors(O, ref.K, dev)
    ws_bytes = workspace_size(problem)
    ws = workspace if workspace is not None else ctx.workspace(ws_bytes)
    _check(load_library().fs_certify_lex(ctx.handle, ref.ptr, ivs, O, float(eps), state.data_ptr(),
                                         _alloc_struct(cons), _alloc_struct(opt), gmm.data_ptr(), ggp.data_ptr(),
                                         ws.data_ptr(), ws.numel(), _stream(dev, stream)))
    return CertifyLexOutput(state, gmm, ggp, cons, opt)


@dataclass
class ScoreLexOutput:
    score_maxmin: object   # [O, E] float64
    score_goodput: object  # [O, E] float64
    gap_maxmin: object     # [O] float64
    gap_goodput: object    # [O] float64
    best: object           # [O] int32


def score_lex_workspace_size(problem, n_orders: int, n_cand: int, n_samples: int) -> int:
    ref = _ProblemRef(problem)
    out = ctypes.c_size_t()
    _check(load_library().fs_score_lex_workspace_size(ref.ptr, int(n_orders), int(n_cand), int(n_samples),
                                                      ctypes.byref(out)))
    return int(out.value)


class ScoreLexPlan:
    """One fs_score_candidates_lex call with its arguments checked and
    marshalled once; run() enqueues the call again on the same device
    buffers.  Shapes as in ScorePlan."""

    def __init__(self, ctx: Context, problem, iv: DeviceIntervals, cand, cap_s, tail_s, stream=None,
                 workspace=None):
        torch = _torch()
        self._ref = _ProblemRef(problem)
        O = int(iv.cap_lo.shape[0])
        E = int(cand.shape[0])
        S = int(cap_s.shape[2]) if E > 0 else 0
        dev = iv.cap_lo.device
        self._ivs = _intervals_struct(iv, O, self._ref.N)
        pcand = _dev_ptr(cand, torch.int32, (E,), "cand")
        pcs = _dev_ptr(cap_s, torch.float32, (O, E, S), "cap_s")
        pts = _dev_ptr(tail_s, torch.float32, (O, E, S), "tail_s")
        out = ScoreLexOutput(torch.empty((O, E), dtype=torch.float64, device=dev),
                             torch.empty((O, E), dtype=torch.float64, device=dev),
                             torch.empty(O, dtype=torch.float64, device=dev),
                             torch.empty(O, dtype=torch.float64, device=dev),
                             torch.empty(O, dtype=torch.int32, device=dev))
        ws_bytes = score_lex_workspace_size(problem, O, E, S)
        ws = workspace if workspace is not None else ctx.workspace(ws_bytes)
        self.out, self._ws, self._keep = out, ws, (iv, cand, cap_s, tail_s)
        self._fn = load_library().fs_score_candidates_lex
        self._args = (ctx.handle, self._ref.ptr, self._ivs, O, pcand, E, pcs, pts, S,
                      out.score_maxmin.data_ptr(), out.score_goodput.data_ptr(), out.gap_maxmin.data_ptr(),
                      out.gap_goodput.data_ptr(), out.best.data_ptr(), ws.data_ptr(), ws.numel(),
                      _stream(dev, stream))

    def run(self) -> ScoreLexOutput:
        _check(self._fn(*self._args))
        return self.out


def score_candidates_lex(ctx: Context, problem, iv: DeviceIntervals, cand, cap_s, tail_s, stream=None,
                         workspace=None) -> ScoreLexOutput:
    """The stage-wise score under the whole objective
    (fs_score_candidates_lex); shapes as in score_candidates."""
    return ScoreLexPlan(ctx, problem, iv, cand, cap_s, tail_s, stream, workspace).run()


def refit_intervals(ctx: Context, problem, iv: DeviceIntervals, stream=None) -> DeviceIntervals:
    """Algorithm 1's fit step (fs_refit_intervals) on [O, N] device
    intervals; returns new intervals (cap_hi and measured shared with iv)."""
    torch = _torch()
    ref = _ProblemRef(problem)
    O = int(iv.cap_lo.shape[0])
    ivs = _intervals_struct(iv, O, ref.N)
    out = DeviceIntervals(torch.empty_like(iv.cap_lo), iv.cap_hi, torch.empty_like(iv.tail_lo),
                          torch.empty_like(iv.tail_hi), iv.measured)
    _check(load_library().fs_refit_intervals(ctx.handle, ref.ptr, ivs, O, out.cap_lo.data_ptr(),
                                             out.tail_lo.data_ptr(), out.tail_hi.data_ptr(),
                                             _stream(iv.cap_lo.device, stream)))
    return out


def clamp_samples(ctx: Context, problem, iv: DeviceIntervals, cand, cap_s, tail_s, stream=None):
    """The candidates' samples clamped into their current intervals
    (fs_clamp_samples); returns new (cap_s, tail_s) tensors [O, E, S]."""
    torch = _torch()
    ref = _ProblemRef(problem)
    O = int(iv.cap_lo.shape[0])
    E = int(cand.shape[0])
    S = int(cap_s.shape[2]) if E > 0 else 0
    ivs = _intervals_struct(iv, O, ref.N)
    pcand = _dev_ptr(cand, torch.int32, (E,), "cand")
    pcs = _dev_ptr(cap_s, torch.float32, (O, E, S), "cap_s")
    pts = _dev_ptr(tail_s, torch.float32, (O, E, S), "tail_s")
    cs_out, ts_out = torch.empty_like(cap_s), torch.empty_like(tail_s)
    _check(load_library().fs_clamp_samples(ctx.handle, ref.ptr, ivs, O, pcand, E, pcs, pts, S, cs_out.data_ptr(),
                                           ts_out.data_ptr(), _stream(iv.cap_lo.device, stream)))
    return cs_out, ts_out


def loop_refit_workspace_size(problem, n_orders: int, n_cand: int, n_samples: int) -> int:
    ref = _ProblemRef(problem)
    out = ctypes.c_size_t()
    _check(load_library().fs_loop_refit_workspace_size(ref.ptr, int(n_orders), int(n_cand), int(n_samples),
                                                       ctypes.byref(out)))
    return int(out.value)


def loop_workspace_size(problem, n_orders: int, n_cand: int, n_samples: int) -> int:
    ref = _ProblemRef(problem)
    out = ctypes.c_size_t()
    _check(load_library().fs_loop_workspace_size(ref.ptr, int(n_orders), int(n_cand), int(n_samples),
                                                 ctypes.byref(out)))
    return int(out.value)


@dataclass
class LoopOutput:
    state: object        # [O] int32
    finished: object     # [O] uint8
    rounds: object       # [O] int32
    gpu_seconds: object  # [O] float64
    reveals: object      # [O, max_rounds] int32
    final: dict          # [O] allocation tensors (objective, tp_index, replicas, floors_met, goodput)
    tau_truth: object    # [O] float32
    tau_oracle: object   # [O] float32


def profile_loop(ctx: Context, problem, iv: DeviceIntervals, truth_cap, truth_tail, cand, cap_s, tail_s,
                 eps: float = 0.05, policy: int = POLICY_SCORE, order=None, max_rounds: int | None = None,
                 check_every: int = 4, stream=None, workspace=None, refit: bool = False) -> LoopOutput:
    """The profiling loop (fs_profile_loop) for O trajectories.  iv holds
    the initial designs [O, N]; truth_cap / truth_tail are float32 [O, N]
    device tensors; order is an int32 [O, E] device tensor (policy
    POLICY_ORDER) or None.  max_rounds defaults to E."""
    torch = _torch()
    ref = _ProblemRef(problem)
    O = int(iv.cap_lo.shape[0])
    E = int(cand.shape[0])
    S = int(cap_s.shape[2]) if (E > 0 and policy == POLICY_SCORE) else 0
    R = E if max_rounds is None else int(max_rounds)
    dev = iv.cap_lo.device
    ivs = _intervals_struct(iv, O, ref.N)
    ptc = _dev_ptr(truth_cap, torch.float32, (O, ref.N), "truth_cap")
    ptt = _dev_ptr(truth_tail, torch.float32, (O, ref.N), "truth_tail")
    pcand = _dev_ptr(cand, torch.int32, (E,), "cand")
    pcs = _dev_ptr(cap_s, torch.float32, (O, E, S), "cap_s") if S else None
    pts = _dev_ptr(tail_s, torch.float32, (O, E, S), "tail_s") if S else None
    pord = _dev_ptr(order, torch.int32, (O, E), "order") if order is not None else None
    out = LoopOutput(torch.empty(O, dtype=torch.int32, device=dev), torch.empty(O, dtype=torch.uint8, device=dev),
                     torch.empty(O, dtype=torch.int32, device=dev), torch.empty(O, dtype=torch.float64, device=dev),
                     torch.empty((O, R), dtype=torch.int32, device=dev), _alloc_tensors(O, ref.K, dev),
                     torch.empty(O, dtype=torch.float32, device=dev), torch.empty(O, dtype=torch.float32, device=dev))
    lo = _LoopOut(out.state.data_ptr(), out.finished.data_ptr(), out.rounds.data_ptr(), out.gpu_seconds.data_ptr(),
                  out.reveals.data_ptr() if R > 0 else None, _alloc_struct(out.final), out.tau_truth.data_ptr(),
                  out.tau_oracle.data_ptr())
    ws_bytes = (loop_refit_workspace_size if refit else loop_workspace_size)(problem, O, E, S)
    ws = workspace if workspace is not None else ctx.workspace(ws_bytes)
    ctx.set_option(OPT_LOOP_REFIT, 1 if refit else 0)
    _check(load_library().fs_profile_loop(ctx.handle, ref.ptr, ivs, O, ptc, ptt, pcand, E, pcs, pts, S,
                                          float(eps), int(policy), pord, R, int(check_every), lo, ws.data_ptr(),
                                          ws.numel(), _stream(dev, stream)))
    return out


class _PolicyRef:
    """Host copy of a class policy (limit [K][M], success_min [K] or None)."""

    def __init__(self, policy, K):
        self.limit = np.ascontiguousarray(np.asarray(policy.limit, dtype=np.float32).reshape(K, -1))
        sm = getattr(policy, "success_min", None)
        self.smin = None if sm is None else np.ascontiguousarray(sm, dtype=np.float32)
        self.M = int(self.limit.shape[1])
        self.s = _SloPolicy(self.M, self.limit.ctypes.data, None if self.smin is None else self.smin.ctypes.data)

    @property
    def ptr(self):
        return ctypes.byref(self.s)


class ReducePlan:
    """One fs_reduce_cells or fs_reduce_samples call with its arguments
    checked and marshalled once; run() enqueues it again on the same device
    buffers."""

    def __init__(self, fn, args, out, keep):
        self._fn, self._args, self.out, self._keep = fn, args, out, keep

    def run(self):
        _check(self._fn(*self._args))
        return self.out

    @staticmethod
    def cells(ctx: Context, problem, policy, tails, success=None, out=None, stream=None) -> "ReducePlan":
        """tails float32 [R, N, M], success float32 [R, N] or None, out [R, N]."""
        torch = _torch()
        ref = _ProblemRef(problem)
        pol = _PolicyRef(policy, ref.K)
        R = int(tails.shape[0])
        dev = tails.device
        pt = _dev_ptr(tails, torch.float32, (R, ref.N, pol.M), "tails")
        ps = _dev_ptr(success, torch.float32, (R, ref.N), "success") if success is not None else None
        if out is None:
            out = torch.empty((R, ref.N), dtype=torch.float32, device=dev)
        po = _dev_ptr(out, torch.float32, (R, ref.N), "out")
        return ReducePlan(load_library().fs_reduce_cells,
                          (ctx.handle, ref.ptr, pol.ptr, pt, ps, R, po, _stream(dev, stream)),
                          out, (ref, pol, tails, success))

    @staticmethod
    def samples(ctx: Context, problem, policy, cand, tail_s, succ_s=None, out=None, stream=None) -> "ReducePlan":
        """cand int32 [E], tail_s float32 [O, E, S, M], succ_s [O, E, S] or None, out [O, E, S]."""
        torch = _torch()
        ref = _ProblemRef(problem)
        pol = _PolicyRef(policy, ref.K)
        O, E, S = (int(x) for x in tail_s.shape[:3])
        dev = tail_s.device
        pc = _dev_ptr(cand, torch.int32, (E,), "cand")
        pt = _dev_ptr(tail_s, torch.float32, (O, E, S, pol.M), "tail_s")
        ps = _dev_ptr(succ_s, torch.float32, (O, E, S), "succ_s") if succ_s is not None else None
        if out is None:
            out = torch.empty((O, E, S), dtype=torch.float32, device=dev)
        po = _dev_ptr(out, torch.float32, (O, E, S), "out")
        return ReducePlan(load_library().fs_reduce_samples,
                          (ctx.handle, ref.ptr, pol.ptr, pc, E, pt, ps, O, S, po, _stream(dev, stream)),
                          out, (ref, pol, cand, tail_s, succ_s))


def reduce_cells(ctx: Context, problem, policy, tails, success=None, out=None, stream=None):
    """Pseudo-tails of cells under a class policy (fs_reduce_cells): tails is
    a float32 [R, N, M] device tensor, success float32 [R, N] or None;
    returns float32 [R, N] holding 0 (feasible) or +inf."""
    return ReducePlan.cells(ctx, problem, policy, tails, success, out, stream).run()


def reduce_samples(ctx: Context, problem, policy, cand, tail_s, succ_s=None, out=None, stream=None):
    """Pseudo-tails of candidate samples (fs_reduce_samples): tail_s is a
    float32 [O, E, S, M] device tensor, succ_s float32 [O, E, S] or None;
    returns float32 [O, E, S]."""
    return ReducePlan.samples(ctx, problem, policy, cand, tail_s, succ_s, out, stream).run()
