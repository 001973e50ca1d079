"""Active-set batched entropic-OT Sinkhorn for MI355X (gfx950).

Thin Python binding of the C ABI in ``include/ds.h``: this module only
marshals torch tensors (device memory and the current HIP stream) into the
library's structs. Every step of the solve runs in the library's HIP kernels;
there is no Python or CPU fallback -- if the built library is missing the call
fails loudly.

    f, g, depth, residual, status, order = solve(X, Y, a, b, eps, tol)

solves W independent problems (eq:eot of arxiv 2607.24741, Sec. 2) by
log-domain Sinkhorn (eq:sinkhorn-cycle), stopping each lane at its first audit
with max(||pi 1 - a||_1, ||pi^T 1 - b||_1) <= tol (eq:release-contract) and
removing finished lanes from the packed batch (Sec. 3.2).
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

__all__ = ["solve", "solve_noalloc", "workspace_bytes", "load_library", "library_path", "DSError",
           "MODES", "LANE_CONVERGED", "LANE_MAX_ITER", "LANE_NONFINITE",
           "F_SHADOW", "F_TIMING", "F_FORCE_VALU", "F_FORCE_MFMA", "F_PRECISE",
           "F_MATERIALIZE", "F_GUARD", "F_FAST32", "F_MATRIX_FREE"]

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIBPATH = os.path.join(_PKG, "_lib", "libdrainsinkhorn.so")
API_VERSION = 4   # the structs below mirror include/ds.h at this version

MODES = {"active": 0, "static": 1, "logical": 2}
LANE_CONVERGED, LANE_MAX_ITER, LANE_NONFINITE = 0, 1, 2
F_SHADOW, F_TIMING, F_FORCE_VALU, F_FORCE_MFMA, F_PRECISE, F_MATERIALIZE, F_GUARD = 1, 2, 4, 8, 16, 32, 64
F_FAST32 = 128   # float32 state on the matrix cores (d <= 16); default: float64 state
F_MATRIX_FREE = 256   # d > 32: K-looped matrix-core half-step instead of the materialised cost

_ERRS = {0: "DS_OK", 1: "DS_E_INVALID", 2: "DS_E_WORKSPACE", 3: "DS_E_HIP",
         4: "DS_E_UNSUPPORTED", 5: "DS_E_INTERNAL"}


class DSError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{_ERRS.get(code, code)}: {msg}")
        self.code = code


class _Problem(ctypes.Structure):
    _fields_ = [("W", ctypes.c_int32), ("n_max", ctypes.c_int32), ("m_max", ctypes.c_int32),
                ("d", ctypes.c_int32), ("X", ctypes.c_void_p), ("Y", ctypes.c_void_p),
                ("a", ctypes.c_void_p), ("b", ctypes.c_void_p), ("eps", ctypes.c_void_p),
                ("n", ctypes.c_void_p), ("m", ctypes.c_void_p), ("g0", ctypes.c_void_p)]


class _Options(ctypes.Structure):
    _fields_ = [("tol", ctypes.c_float), ("screen_tol", ctypes.c_float),
                ("max_iter", ctypes.c_int32), ("audit_every", ctypes.c_int32),
                ("mode", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("streams", ctypes.c_int32)]


class _Result(ctypes.Structure):
    _fields_ = [("f", ctypes.c_void_p), ("g", ctypes.c_void_p), ("depth", ctypes.c_void_p),
                ("residual", ctypes.c_void_p), ("row_residual", ctypes.c_void_p),
                ("col_residual", ctypes.c_void_p), ("status", ctypes.c_void_p),
                ("order", ctypes.c_void_p)]


class _Stats(ctypes.Structure):
    _fields_ = [("slots_update", ctypes.c_int64), ("halfsteps_executed", ctypes.c_int64),
                ("pair_evals", ctypes.c_int64), ("check_pair_evals", ctypes.c_int64),
                ("bytes_compacted", ctypes.c_int64),
                ("l_max", ctypes.c_int32), ("cycles", ctypes.c_int32),
                ("audits", ctypes.c_int32), ("screen_positive", ctypes.c_int32),
                ("check_failures", ctypes.c_int32), ("compactions", ctypes.c_int32),
                ("missed_ready", ctypes.c_int32), ("update_launches", ctypes.c_int32),
                ("ms_total", ctypes.c_double), ("ms_update", ctypes.c_double),
                ("timed_pair_evals", ctypes.c_int64),
                ("ms_check", ctypes.c_double), ("ms_compact", ctypes.c_double),
                ("width_trace", ctypes.POINTER(ctypes.c_int32)),
                ("width_trace_len", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_size_t), ("sub_batches", ctypes.c_int32),
                ("screen_discrepancy", ctypes.c_double), ("guard_missed", ctypes.c_int32)]


_lib = None


def library_path() -> str:
    return _LIBPATH


def load_library():
    """Load the built HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIBPATH):
        raise RuntimeError(
            f"HIP library not built: {_LIBPATH} is missing. Run "
            "`python -m paper_2607_24741_amd.build` (or __graft_entry__.build()).")
    lib = ctypes.CDLL(_LIBPATH)
    lib.ds_api_version.restype = ctypes.c_int
    if lib.ds_api_version() != API_VERSION:
        raise RuntimeError(f"{_LIBPATH} implements ABI version {lib.ds_api_version()}, this "
                           f"binding expects {API_VERSION}: rebuild the library")
    lib.ds_workspace_bytes.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Options),
                                       ctypes.POINTER(ctypes.c_size_t)]
    lib.ds_workspace_bytes.restype = ctypes.c_int
    lib.ds_solve.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Options),
                             ctypes.POINTER(_Result), ctypes.c_void_p, ctypes.c_size_t,
                             ctypes.c_void_p, ctypes.POINTER(_Stats)]
    lib.ds_solve.restype = ctypes.c_int
    lib.ds_solve_noalloc.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Options),
                                     ctypes.POINTER(_Result), ctypes.c_void_p,
                                     ctypes.POINTER(_Stats)]
    lib.ds_solve_noalloc.restype = ctypes.c_int
    lib.ds_error_string.argtypes = [ctypes.c_int]
    lib.ds_error_string.restype = ctypes.c_char_p
    lib.ds_last_error_message.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(lib, code):
    if code != 0:
        raise DSError(code, lib.ds_last_error_message().decode())


def _options(tol, screen_tol, max_iter, audit_every, mode, flags, streams=0):
    if mode not in MODES:
        raise ValueError(f"mode must be one of {sorted(MODES)}")
    return _Options(tol=float(tol), screen_tol=float(screen_tol or 0.0), max_iter=int(max_iter),
                    audit_every=int(audit_every), mode=MODES[mode], flags=int(flags),
                    streams=int(streams))


def workspace_bytes(W, n_max, m_max, d, *, tol=1e-3, max_iter=5000, audit_every=1,
                    mode="active", flags=0, streams=0) -> int:
    lib = load_library()
    pr = _Problem(W=W, n_max=n_max, m_max=m_max, d=d)
    op = _options(tol, None, max_iter, audit_every, mode, flags, streams)
    out = ctypes.c_size_t(0)
    _check(lib, lib.ds_workspace_bytes(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(out)))
    return int(out.value)


@dataclass
class Stats:
    slots_update: int
    halfsteps_executed: int
    pair_evals: int
    check_pair_evals: int
    bytes_compacted: int
    l_max: int
    cycles: int
    audits: int
    screen_positive: int
    check_failures: int
    compactions: int
    missed_ready: int
    update_launches: int
    ms_total: float
    ms_update: float
    timed_pair_evals: int
    ms_check: float
    ms_compact: float
    width_trace: list
    workspace_bytes: int
    sub_batches: int
    screen_discrepancy: float
    guard_missed: int
    row_residual: object = None   # [W] tensor
    col_residual: object = None   # [W] tensor


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


_OUT_REQUIRED = ("f", "g", "depth", "residual", "status")
_OUT_OPTIONAL = ("row_residual", "col_residual", "order")


def _check_out(out, W, n_max, m_max, dev):
    """Validates caller-provided output tensors (the library writes through
    their raw pointers): f [W, n_max] and g [W, m_max] float32, depth and
    status int32 [W], residual float32 [W]; row_residual / col_residual
    (float32 [W]) and order (int32 [W]) may be absent or None."""
    import torch
    spec = dict(f=(torch.float32, (W, n_max)), g=(torch.float32, (W, m_max)),
                depth=(torch.int32, (W,)), residual=(torch.float32, (W,)),
                row_residual=(torch.float32, (W,)), col_residual=(torch.float32, (W,)),
                status=(torch.int32, (W,)), order=(torch.int32, (W,)))
    unknown = set(out) - set(spec)
    if unknown:
        raise ValueError(f"unknown output(s) {sorted(unknown)}")
    checked = {}
    for k, (dt, shape) in spec.items():
        t = out.get(k)
        if t is None:
            if k in _OUT_REQUIRED:
                raise ValueError(f"output {k} is required")
            checked[k] = None
            continue
        if t.dtype != dt or not t.is_contiguous() or t.device != dev or tuple(t.shape) != shape:
            raise ValueError(f"output {k} must be a contiguous {dt} tensor of shape {shape} on {dev}")
        checked[k] = t
    return checked


def solve_noalloc(X, Y, a, b, eps, tol, *, out, n=None, m=None, g0=None, max_iter=5000,
                  audit_every=1, mode="active", screen_tol=None, flags=0, return_stats=False,
                  trace_len=0):
    """``solve`` through ds_solve_noalloc: the workspace is the library's fixed
    per-GPU array (64 MiB), one sub-batch on the current stream, and the caller
    passes every output tensor (``out``, as for ``solve``), so that neither
    the library nor this binding allocates device memory for the call."""
    return solve(X, Y, a, b, eps, tol, n=n, m=m, g0=g0, max_iter=max_iter,
                 audit_every=audit_every, mode=mode, screen_tol=screen_tol, flags=flags,
                 streams=1, return_stats=return_stats, trace_len=trace_len, out=out,
                 _noalloc=True)


def solve(X, Y, a, b, eps, tol, *, n=None, m=None, g0=None, max_iter=5000, audit_every=1,
          mode="active", screen_tol=None, flags=0, streams=0, return_stats=False,
          workspace=None, trace_len=0, out=None, _noalloc=False):
    """Solve W independent entropic OT problems on the current GPU.

    X [W, n_max, d], Y [W, m_max, d], a [W, n_max], b [W, m_max], eps [W]:
    contiguous float32 CUDA tensors; n, m optional int32 [W] valid prefixes;
    g0 an optional float32 [W, m_max] proposal (initial target potential;
    default: the cold proposal g^0 = 0).
    Returns (f, g, depth, residual, status, order) and, with
    ``return_stats=True``, a Stats record as well. ``workspace`` may be a
    pre-allocated uint8 CUDA tensor of at least ``workspace_bytes(...)``.
    """
    import torch
    lib = load_library()
    W, n_max, d = X.shape
    m_max = Y.shape[1]
    dev = X.device
    if dev.type != "cuda":
        raise ValueError("inputs must be CUDA (HIP) tensors")
    for name, t, shape in (("X", X, (W, n_max, d)), ("Y", Y, (W, m_max, d)), ("a", a, (W, n_max)),
                           ("b", b, (W, m_max)), ("eps", eps, (W,)), ("g0", g0, (W, m_max))):
        if t is None and name == "g0":
            continue
        if t.dtype != torch.float32 or not t.is_contiguous() or t.device != dev:
            raise ValueError(f"{name} must be a contiguous float32 tensor on {dev}")
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {shape}")
    for name, t in (("n", n), ("m", m)):
        if t is not None and (t.dtype != torch.int32 or not t.is_contiguous() or t.device != dev
                              or tuple(t.shape) != (W,)):
            raise ValueError(f"{name} must be a contiguous int32 tensor of shape ({W},) on {dev}")
    pr = _Problem(W=W, n_max=n_max, m_max=m_max, d=d, X=_ptr(X), Y=_ptr(Y), a=_ptr(a),
                  b=_ptr(b), eps=_ptr(eps), n=_ptr(n), m=_ptr(m), g0=_ptr(g0))
    op = _options(tol, screen_tol, max_iter, audit_every, mode, flags, streams)
    if _noalloc:
        if out is None:
            raise ValueError("solve_noalloc needs caller-provided outputs (out=...)")
        out = _check_out(out, W, n_max, m_max, dev)
        res = _Result(**{k: _ptr(v) for k, v in out.items()})
        st = _Stats()
        trace_buf = None
        if trace_len:
            trace_buf = (ctypes.c_int32 * int(trace_len))()
            st.width_trace = ctypes.cast(trace_buf, ctypes.POINTER(ctypes.c_int32))
            st.width_trace_len = int(trace_len)
        stream = torch.cuda.current_stream(dev).cuda_stream
        with torch.cuda.device(dev):
            code = lib.ds_solve_noalloc(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(res),
                                        ctypes.c_void_p(stream), ctypes.byref(st))
        _check(lib, code)
        return _returns(out, st, trace_buf, return_stats)
    need = ctypes.c_size_t(0)
    _check(lib, lib.ds_workspace_bytes(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(need)))
    if workspace is None:
        workspace = torch.empty(int(need.value) + 256, dtype=torch.uint8, device=dev)
    elif (workspace.dtype != torch.uint8 or not workspace.is_contiguous()
          or workspace.device != dev):
        raise ValueError(f"workspace must be a contiguous uint8 tensor on {dev}")
    base = workspace.data_ptr()
    shift = (-base) % 256
    if workspace.numel() - shift < int(need.value):
        raise ValueError(f"workspace holds {workspace.numel()} bytes ({shift} of them before the "
                         f"first 256-byte boundary); the call needs {int(need.value)} from there")
    ws_ptr, ws_bytes = base + shift, workspace.numel() - shift
    if out is None:
        out = dict(f=torch.empty((W, n_max), dtype=torch.float32, device=dev),
                   g=torch.empty((W, m_max), dtype=torch.float32, device=dev),
                   depth=torch.empty(W, dtype=torch.int32, device=dev),
                   residual=torch.empty(W, dtype=torch.float32, device=dev),
                   row_residual=torch.empty(W, dtype=torch.float32, device=dev),
                   col_residual=torch.empty(W, dtype=torch.float32, device=dev),
                   status=torch.empty(W, dtype=torch.int32, device=dev),
                   order=torch.empty(W, dtype=torch.int32, device=dev))
    else:
        out = _check_out(out, W, n_max, m_max, dev)
    res = _Result(**{k: _ptr(v) for k, v in out.items()})
    st = _Stats()
    trace_buf = None
    if trace_len:
        trace_buf = (ctypes.c_int32 * int(trace_len))()
        st.width_trace = ctypes.cast(trace_buf, ctypes.POINTER(ctypes.c_int32))
        st.width_trace_len = int(trace_len)
    stream = torch.cuda.current_stream(dev).cuda_stream
    with torch.cuda.device(dev):
        code = lib.ds_solve(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(res),
                            ctypes.c_void_p(ws_ptr), ctypes.c_size_t(ws_bytes),
                            ctypes.c_void_p(stream), ctypes.byref(st))
    _check(lib, code)
    return _returns(out, st, trace_buf, return_stats)


def _returns(out, st, trace_buf, return_stats):
    ret = (out["f"], out["g"], out["depth"], out["residual"], out["status"], out.get("order"))
    if not return_stats:
        return ret
    wt = list(trace_buf[:st.width_trace_len]) if trace_buf is not None else []
    stats = Stats(st.slots_update, st.halfsteps_executed, st.pair_evals, st.check_pair_evals,
                  st.bytes_compacted,
                  st.l_max, st.cycles, st.audits, st.screen_positive, st.check_failures,
                  st.compactions, st.missed_ready, st.update_launches, st.ms_total, st.ms_update,
                  st.timed_pair_evals, st.ms_check, st.ms_compact, wt, st.workspace_bytes,
                  st.sub_batches, st.screen_discrepancy, st.guard_missed,
                  out.get("row_residual"), out.get("col_residual"))
    return ret + (stats,)
