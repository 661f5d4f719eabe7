"""ctypes binding of libturbomuon.so: argument marshalling only.

Every step of the orthogonalization runs in the library's HIP kernels; this
module checks tensor metadata, passes raw device pointers, the coefficient
table and the current HIP stream, and turns status codes into exceptions.
It never computes anything itself and has no fallback: a missing library is
an error.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libturbomuon.so")

TM_OK = 0
TM_ERR_INVALID_ARG = -1
TM_ERR_UNSUPPORTED = -2
TM_ERR_NO_MEMORY = -3
TM_ERR_HIP = -4

PRECOND = {"none": 0, "frobenius": 1, "frob": 1, "aol": 2, "schatten4": 3, "s4": 3}
PHASES = {"transpose_in": 0, "frob": 1, "gram": 2, "aol_vector": 3, "poly": 4, "update": 5,
          "apply_scale": 6, "copy_out": 7, "load_in": 8, "scale_a": 9, "opt_momentum": 10,
          "opt_apply": 11, "fused": 12}
TM_MAX_DIM = 65536
TM_MAX_ITERS = 64

_c_i64p = ctypes.POINTER(ctypes.c_int64)
_c_fp = ctypes.POINTER(ctypes.c_float)

_SIGNATURES = {
    "tm_orthogonalize": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                        ctypes.c_int64, ctypes.c_int, _c_fp, ctypes.c_int,
                                        ctypes.c_void_p]),
    "tm_orthogonalize_f32": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                            ctypes.c_int64, ctypes.c_int, _c_fp, ctypes.c_int,
                                            ctypes.c_void_p]),
    "tm_orthogonalize_grouped": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p), _c_i64p, _c_i64p,
                                                ctypes.c_int64, ctypes.c_int, _c_fp, ctypes.c_int,
                                                ctypes.c_void_p]),
    "tm_orthogonalize_grouped_f32": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p), _c_i64p,
                                                    _c_i64p, ctypes.c_int64, ctypes.c_int, _c_fp,
                                                    ctypes.c_int, ctypes.c_void_p]),
    "tm_muon_step_grouped": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p),
                                            ctypes.POINTER(ctypes.c_void_p),
                                            ctypes.POINTER(ctypes.c_void_p), _c_i64p, _c_i64p,
                                            ctypes.c_int64, ctypes.c_float, ctypes.c_float,
                                            ctypes.c_int, ctypes.c_float, ctypes.c_int,
                                            ctypes.c_int, _c_fp, ctypes.c_int, ctypes.c_void_p]),
    "tm_orthogonalize_noalloc": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                                ctypes.c_int64, ctypes.c_int, _c_fp, ctypes.c_int,
                                                ctypes.c_void_p]),
    "tm_schedule_tail": (_c_fp, [_c_fp, ctypes.c_int, ctypes.c_int]),
    "tm_workspace_bytes": (ctypes.c_uint64, [_c_i64p, _c_i64p, ctypes.c_int64, ctypes.c_int]),
    "tm_release_workspaces": (ctypes.c_int, []),
    "tm_timing_enable": (ctypes.c_int, [ctypes.c_int]),
    "tm_timing_read": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_int64)]),
    "tm_timing_reset": (ctypes.c_int, []),
    "tm_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "tm_last_error": (ctypes.c_char_p, []),
    "tm_version": (ctypes.c_char_p, []),
}

_lib = None


class TurboMuonError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str):
        self.status = status
        super().__init__(f"{fn} failed: {status_string(status)}: {detail}")


def lib() -> ctypes.CDLL:
    """Load libturbomuon.so (built in-tree by paper_2512_04632_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with "
                               "`python -m paper_2512_04632_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().tm_status_string(status).decode()


def last_error() -> str:
    return lib().tm_last_error().decode()


def version() -> str:
    return lib().tm_version().decode()


def _check(fn: str, status: int) -> None:
    if status != TM_OK:
        raise TurboMuonError(fn, status, last_error())


def _coeff_array(iters: int, coeffs):
    if coeffs is None:
        return None
    flat = [float(v) for row in coeffs for v in row]
    if len(flat) != 3 * iters:
        raise ValueError("coeffs must hold one (a, b, c) triple per iteration")
    return (ctypes.c_float * len(flat))(*flat)


def _precond(p) -> int:
    if isinstance(p, int):
        return p
    return PRECOND[p]


def _stream_handle(t, stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(t.device)
    return int(stream.cuda_stream)


def orthogonalize(x, iters: int = 4, coeffs: Optional[Sequence] = None, precond="aol",
                  stream=None):
    """Orthogonalize x in place: (m, n) or (batch, m, n), contiguous, bf16 or fp32, on a GPU.

    iters Newton-Schulz iterations after the pre-conditioning ("aol",
    "frobenius", "schatten4" or "none"); coeffs is an optional list of (a, b, c) per
    iteration.  Work is enqueued on `stream` (default: the current stream).
    Returns x.
    """
    import torch
    if not x.is_cuda:
        raise ValueError("x must be a device tensor")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    if x.dim() not in (2, 3):
        raise ValueError("x must be (m, n) or (batch, m, n)")
    if x.dtype == torch.bfloat16:
        fn = "tm_orthogonalize"
    elif x.dtype == torch.float32:
        fn = "tm_orthogonalize_f32"
    else:
        raise ValueError("x must be bfloat16 or float32")
    m, n = int(x.shape[-2]), int(x.shape[-1])
    batch = int(x.shape[0]) if x.dim() == 3 else 1
    carr = _coeff_array(iters, coeffs)
    with torch.cuda.device(x.device):
        st = getattr(lib(), fn)(ctypes.c_void_p(x.data_ptr()), m, n, batch, int(iters),
                                carr, _precond(precond), ctypes.c_void_p(_stream_handle(x, stream)))
    _check(fn, st)
    return x


TM_NOALLOC_SCRATCH_BYTES = 64 << 20


def orthogonalize_noalloc(x, iters: int = 4, coeffs: Optional[Sequence] = None, precond="aol",
                          stream=None):
    """tm_orthogonalize_noalloc: as orthogonalize for a bf16 (m, n) or (batch, m, n)
    tensor, with the workspace in the library's static per-GPU scratch array instead
    of an allocated one (raises TurboMuonError if the call needs more).  Returns x."""
    import torch
    if not x.is_cuda or not x.is_contiguous() or x.dim() not in (2, 3):
        raise ValueError("x must be a contiguous (m, n) or (batch, m, n) device tensor")
    if x.dtype != torch.bfloat16:
        raise ValueError("x must be bfloat16")
    m, n = int(x.shape[-2]), int(x.shape[-1])
    batch = int(x.shape[0]) if x.dim() == 3 else 1
    carr = _coeff_array(iters, coeffs)
    with torch.cuda.device(x.device):
        st = lib().tm_orthogonalize_noalloc(ctypes.c_void_p(x.data_ptr()), m, n, batch,
                                            int(iters), carr, _precond(precond),
                                            ctypes.c_void_p(_stream_handle(x, stream)))
    _check("tm_orthogonalize_noalloc", st)
    return x


def orthogonalize_grouped(xs: Sequence, iters: int = 4, coeffs: Optional[Sequence] = None,
                          precond="aol", stream=None):
    """Orthogonalize a list of 2-D tensors (any shapes, one dtype, one device) in place."""
    import torch
    xs = list(xs)
    if not xs:
        return xs
    dt, dev = xs[0].dtype, xs[0].device
    for t in xs:
        if not t.is_cuda or t.dim() != 2 or not t.is_contiguous():
            raise ValueError("grouped inputs must be contiguous 2-D device tensors")
        if t.dtype != dt or t.device != dev:
            raise ValueError("grouped inputs must share dtype and device")
    if dt == torch.bfloat16:
        fn = "tm_orthogonalize_grouped"
    elif dt == torch.float32:
        fn = "tm_orthogonalize_grouped_f32"
    else:
        raise ValueError("inputs must be bfloat16 or float32")
    cnt = len(xs)
    ptrs = (ctypes.c_void_p * cnt)(*[t.data_ptr() for t in xs])
    ms = (ctypes.c_int64 * cnt)(*[int(t.shape[0]) for t in xs])
    ns = (ctypes.c_int64 * cnt)(*[int(t.shape[1]) for t in xs])
    carr = _coeff_array(iters, coeffs)
    with torch.cuda.device(dev):
        st = getattr(lib(), fn)(ptrs, ms, ns, cnt, int(iters), carr, _precond(precond),
                                ctypes.c_void_p(_stream_handle(xs[0], stream)))
    _check(fn, st)
    return xs


def muon_step_grouped(params: Sequence, grads: Sequence, bufs: Sequence, lr: float,
                      momentum: float = 0.95, nesterov: bool = True, weight_decay: float = 0.0,
                      shape_scale: bool = True, iters: int = 4, coeffs: Optional[Sequence] = None,
                      precond="aol", stream=None):
    """One optimizer step (tm_muon_step_grouped) over lists of 2-D fp32 device tensors.

    params and bufs (momentum buffers) are updated in place; grads are read.
    """
    import torch
    params, grads, bufs = list(params), list(grads), list(bufs)
    if not (len(params) == len(grads) == len(bufs)):
        raise ValueError("params, grads and bufs must have the same length")
    if not params:
        return
    dev = params[0].device
    for w, g, m in zip(params, grads, bufs):
        for t in (w, g, m):
            if (not t.is_cuda or t.dtype != torch.float32 or t.dim() != 2 or
                    not t.is_contiguous() or t.device != dev):
                raise ValueError("optimizer tensors must be contiguous 2-D fp32 tensors on one device")
        if g.shape != w.shape or m.shape != w.shape:
            raise ValueError("gradient and momentum buffer must match the parameter's shape")
    cnt = len(params)
    W = (ctypes.c_void_p * cnt)(*[t.data_ptr() for t in params])
    G = (ctypes.c_void_p * cnt)(*[t.data_ptr() for t in grads])
    M = (ctypes.c_void_p * cnt)(*[t.data_ptr() for t in bufs])
    ms = (ctypes.c_int64 * cnt)(*[int(t.shape[0]) for t in params])
    ns = (ctypes.c_int64 * cnt)(*[int(t.shape[1]) for t in params])
    carr = _coeff_array(iters, coeffs)
    with torch.cuda.device(dev):
        st = lib().tm_muon_step_grouped(W, G, M, ms, ns, cnt, float(lr), float(momentum),
                                        1 if nesterov else 0, float(weight_decay),
                                        1 if shape_scale else 0, int(iters), carr,
                                        _precond(precond),
                                        ctypes.c_void_p(_stream_handle(params[0], stream)))
    _check("tm_muon_step_grouped", st)


def schedule_tail(schedule: Sequence, iters: int) -> list:
    """The rows of a coefficient schedule that a call with `iters` iterations runs
    (tm_schedule_tail: the last `iters` rows)."""
    flat = [float(v) for row in schedule for v in row]
    rows = len(flat) // 3
    if rows * 3 != len(flat):
        raise ValueError("a schedule holds (a, b, c) triples")
    arr = (ctypes.c_float * max(len(flat), 1))(*flat)
    p = lib().tm_schedule_tail(arr, rows, int(iters))
    if not p:
        raise TurboMuonError("tm_schedule_tail", TM_ERR_INVALID_ARG, last_error())
    return [(p[3 * i], p[3 * i + 1], p[3 * i + 2]) for i in range(int(iters))]


def workspace_bytes(shapes: Sequence, dtype_bytes: int) -> int:
    cnt = len(shapes)
    ms = (ctypes.c_int64 * max(cnt, 1))(*[int(s[0]) for s in shapes])
    ns = (ctypes.c_int64 * max(cnt, 1))(*[int(s[1]) for s in shapes])
    return int(lib().tm_workspace_bytes(ms, ns, cnt, dtype_bytes))


def release_workspaces() -> None:
    _check("tm_release_workspaces", lib().tm_release_workspaces())


def timing_enable(on: bool = True) -> None:
    _check("tm_timing_enable", lib().tm_timing_enable(1 if on else 0))


def timing_reset() -> None:
    _check("tm_timing_reset", lib().tm_timing_reset())


def timing_read(phase: str):
    """(summed event milliseconds, launches) of one phase since the last reset."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check("tm_timing_read", lib().tm_timing_read(PHASES[phase], ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
