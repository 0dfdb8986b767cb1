"""Thin ctypes binding of librecblr.so (the C ABI in include/recblr.h).

Two layers, both pure argument marshalling (every step of the computation runs
in the HIP kernels of librecblr.so):

* ``recblr_*`` functions mirror the C entry points one to one: they take raw
  device pointers (ints) and sizes and return the C status code.
* ``bdlru_scan_forward`` and friends take torch tensors that live on the GPU,
  check their shapes and dtypes, allocate outputs and workspace with torch,
  call the C entry point on the current HIP stream and raise on a non-zero
  status.

There is no fallback: if the library is missing or fails to load, importing
this module raises.  Build it first with ``python -m paper_2406_12580_amd.build``.
"""
from __future__ import annotations

import ctypes
import functools
import inspect
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librecblr.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing; build it with `python -m paper_2406_12580_amd.build`")
_lib = ctypes.CDLL(LIB_PATH)

OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_SCRATCH = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
(OP_SCAN_FORWARD, OP_SCAN_BACKWARD, OP_FORWARD, OP_BACKWARD, OP_STEP, OP_GATED_FORWARD,
 OP_GATED_BACKWARD, OP_SCAN_BACKWARD_METHOD) = range(8)
SCAN_CHUNKED, SCAN_SERIAL, SCAN_TREE = range(3)

EXPORTS = (
    "recblr_status_string", "recblr_workspace_size", "recblr_bdlru_scan_forward",
    "recblr_bdlru_scan_backward", "recblr_bdlru_scan_step", "recblr_bdlru_forward",
    "recblr_bdlru_backward", "recblr_bdlru_step", "recblr_linear_scan_forward",
    "recblr_scan_forward_method", "recblr_scan_backward_method", "recblr_gated_forward", "recblr_bdlru_scan_forward_timed",
    "recblr_bdlru_scan_backward_timed", "recblr_gated_backward", "recblr_model_param_count",
    "recblr_model_param_offsets", "recblr_model_workspace_size", "recblr_blas_create",
    "recblr_blas_destroy", "recblr_model_train_step", "recblr_adam_update",
    "recblr_bdlru_scan_backward_noalloc",
)

_p, _i64, _int, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
_f = ctypes.c_float


class ModelDims(ctypes.Structure):
    """recblr_model_dims."""
    _fields_ = [("B", _i64), ("T", _i64), ("D", _i64), ("E", _i64), ("V", _i64),
                ("layers", _i64), ("K", _int), ("ln_eps", _f)]


class ModelStepOpts(ctypes.Structure):
    """recblr_model_step_opts."""
    _fields_ = [("dropout", _f), ("pad_id", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("offset", ctypes.c_uint64)]


_pd = ctypes.POINTER(ModelDims)
_po = ctypes.POINTER(ModelStepOpts)
_SIGS = {
    "recblr_status_string": ([_int], ctypes.c_char_p),
    "recblr_workspace_size": ([_int, _i64, _i64, _i64, _int], _sz),
    "recblr_bdlru_scan_forward": ([_p] * 7 + [_i64] * 3 + [_int, _p, _sz, _p], _int),
    "recblr_bdlru_scan_backward": ([_p] * 13 + [_i64] * 3 + [_int, _p, _sz, _p], _int),
    "recblr_bdlru_scan_forward_timed": ([_p] * 7 + [_i64] * 3 + [_int, _p, _sz, _p, _p, _p], _int),
    "recblr_bdlru_scan_backward_timed": ([_p] * 13 + [_i64] * 3 + [_int, _p, _sz, _p, _p, _p],
                                         _int),
    "recblr_bdlru_scan_backward_noalloc": ([_p] * 13 + [_i64] * 3 + [_int, _p], _int),
    "recblr_bdlru_scan_step": ([_p] * 6 + [_i64] * 2 + [_int, _p], _int),
    "recblr_bdlru_forward": ([_p] * 9 + [_i64] * 3 + [_int, _p, _sz, _p], _int),
    "recblr_bdlru_backward": ([_p] * 17 + [_i64] * 3 + [_int, _p, _sz, _p], _int),
    "recblr_bdlru_step": ([_p] * 8 + [_i64] * 2 + [_int, _p, _sz, _p], _int),
    "recblr_linear_scan_forward": ([_p] * 5 + [_i64] * 3 + [_p], _int),
    "recblr_scan_forward_method": ([_int] + [_p] * 5 + [_i64] * 3 + [_int, _p, _sz, _p], _int),
    "recblr_scan_backward_method": ([_int] + [_p] * 10 + [_i64] * 3 + [_int, _p, _sz, _p],
                                    _int),
    "recblr_gated_forward": ([_p] * 4 + [_int] + [_p] * 9 + [_i64] * 3 + [_int, _p, _sz, _p],
                             _int),
    "recblr_gated_backward": ([_p] * 4 + [_int] + [_p] * 19 + [_i64] * 3 + [_int, _p, _sz, _p],
                              _int),
    "recblr_model_param_count": ([_pd], _sz),
    "recblr_model_param_offsets": ([_pd, _p, _i64], _i64),
    "recblr_model_workspace_size": ([_pd], _sz),
    "recblr_blas_create": ([ctypes.POINTER(_p)], _int),
    "recblr_blas_destroy": ([_p], _int),
    "recblr_model_train_step": ([_pd, _po] + [_p] * 6 + [_sz, _p, _p], _int),
    "recblr_adam_update": ([_p] * 4 + [_i64, _i64, _f, _f, _f, _f, _p], _int),
}
for _name, (_args, _res) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = _res
    globals()[_name] = _fn


class RecblrError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {recblr_status_string(status).decode()} ({status})")


def _check(status: int, where: str):
    if status != OK:
        raise RecblrError(status, where)


# ------------------------------------------------------------------ torch-level helpers

def io_code(dtype: torch.dtype) -> int:
    if dtype == torch.float32:
        return F32
    if dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported I/O dtype {dtype}; use float32 or bfloat16")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _on_stream(fn):
    """Run a wrapper with its `stream` argument as torch's current stream.

    The workspace and outputs are then allocated by torch's caching allocator
    on the stream the kernels are launched on, so the workspace, released when
    the wrapper returns, is handed out again only to later work on that same
    stream (which runs after the launched kernels).  Without a `stream`
    argument nothing changes: torch's current stream is the launch stream.
    """
    sig = inspect.signature(fn)

    @functools.wraps(fn)
    def wrapper(*args, **kwargs):
        bound = sig.bind(*args, **kwargs)
        s = bound.arguments.get("stream")
        if s is None:
            return fn(*args, **kwargs)
        bound.arguments["stream"] = None
        with torch.cuda.stream(s):
            return fn(*bound.args, **bound.kwargs)
    return wrapper


def _workspace(op: int, B: int, L: int, D: int, io: int, device):
    n = recblr_workspace_size(op, B, L, D, io)
    if n == 0:
        return None, 0
    return torch.empty(n, dtype=torch.uint8, device=device), n


def _f32(t, shape, name):
    if t is None:
        return None
    if t.dtype != torch.float32 or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be float32 of shape {tuple(shape)}")
    return t


def _io(t, shape, dtype, name):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be {dtype} of shape {tuple(shape)}")
    return t


@_on_stream
def bdlru_scan_forward(x, zr, zi, lam, h0=None, stream=None):
    """Gated BD-LRU scan from pre-activations. Returns (h [B,L,D] io, hT [B,D] float32)."""
    B, L, D = x.shape
    io = io_code(x.dtype)
    _io(zr, x.shape, x.dtype, "zr"), _io(zi, x.shape, x.dtype, "zi")
    _f32(lam, (D,), "lambda"), _f32(h0, (B, D), "h0")
    h = torch.empty_like(x)
    hT = torch.empty((B, D), dtype=torch.float32, device=x.device)
    ws, nws = _workspace(OP_SCAN_FORWARD, B, L, D, io, x.device)
    _check(recblr_bdlru_scan_forward(_ptr(x), _ptr(zr), _ptr(zi), _ptr(lam), _ptr(h0), _ptr(h),
                                     _ptr(hT), B, L, D, io, _ptr(ws), nws, _stream(stream)),
           "recblr_bdlru_scan_forward")
    return h, hT


@_on_stream
def bdlru_scan_backward(x, zr, zi, lam, h, dh, h0=None, dhT=None, stream=None):
    """Backward of bdlru_scan_forward. Returns dict dx, dzr, dzi, dlambda, dh0."""
    B, L, D = x.shape
    io = io_code(x.dtype)
    for t, n in ((zr, "zr"), (zi, "zi"), (h, "h"), (dh, "dh")):
        _io(t, x.shape, x.dtype, n)
    _f32(lam, (D,), "lambda"), _f32(h0, (B, D), "h0"), _f32(dhT, (B, D), "dhT")
    out = {k: torch.empty_like(x) for k in ("dx", "dzr", "dzi")}
    out["dlambda"] = torch.empty(D, dtype=torch.float32, device=x.device)
    out["dh0"] = torch.empty((B, D), dtype=torch.float32, device=x.device)
    ws, nws = _workspace(OP_SCAN_BACKWARD, B, L, D, io, x.device)
    _check(recblr_bdlru_scan_backward(
        _ptr(x), _ptr(zr), _ptr(zi), _ptr(lam), _ptr(h0), _ptr(h), _ptr(dh), _ptr(dhT),
        _ptr(out["dx"]), _ptr(out["dzr"]), _ptr(out["dzi"]), _ptr(out["dlambda"]),
        _ptr(out["dh0"]), B, L, D, io, _ptr(ws), nws, _stream(stream)),
        "recblr_bdlru_scan_backward")
    return out


@_on_stream
def bdlru_scan_step(x, zr, zi, lam, h_prev, out=None, stream=None):
    """One recurrent step over [B, D]; returns h_next (float32). out may be h_prev."""
    B, D = x.shape
    io = io_code(x.dtype)
    _io(zr, x.shape, x.dtype, "zr"), _io(zi, x.shape, x.dtype, "zi")
    _f32(lam, (D,), "lambda"), _f32(h_prev, (B, D), "h_prev")
    h_next = torch.empty((B, D), dtype=torch.float32, device=x.device) if out is None else out
    _check(recblr_bdlru_scan_step(_ptr(x), _ptr(zr), _ptr(zi), _ptr(lam), _ptr(h_prev),
                                  _ptr(h_next), B, D, io, _stream(stream)),
           "recblr_bdlru_scan_step")
    return h_next


@_on_stream
def bdlru_forward(x, Wr, br, Wi, bi, lam, h0=None, stream=None):
    """Full forward with gate projections. Returns (h, hT)."""
    B, L, D = x.shape
    io = io_code(x.dtype)
    for t, n in ((Wr, "Wr"), (Wi, "Wi")):
        _io(t, (D, D), x.dtype, n)
    for t, n in ((br, "br"), (bi, "bi")):
        if t is not None:
            _io(t, (D,), x.dtype, n)
    _f32(lam, (D,), "lambda"), _f32(h0, (B, D), "h0")
    h = torch.empty_like(x)
    hT = torch.empty((B, D), dtype=torch.float32, device=x.device)
    ws, nws = _workspace(OP_FORWARD, B, L, D, io, x.device)
    _check(recblr_bdlru_forward(_ptr(x), _ptr(Wr), _ptr(br), _ptr(Wi), _ptr(bi), _ptr(lam),
                                _ptr(h0), _ptr(h), _ptr(hT), B, L, D, io, _ptr(ws), nws,
                                _stream(stream)), "recblr_bdlru_forward")
    return h, hT


@_on_stream
def bdlru_backward(x, Wr, br, Wi, bi, lam, h, dh, h0=None, dhT=None, stream=None):
    """Full backward. Returns dict dx, dWr, dbr, dWi, dbi, dlambda, dh0."""
    B, L, D = x.shape
    io = io_code(x.dtype)
    for t, n in ((Wr, "Wr"), (Wi, "Wi")):
        _io(t, (D, D), x.dtype, n)
    _io(h, x.shape, x.dtype, "h"), _io(dh, x.shape, x.dtype, "dh")
    _f32(lam, (D,), "lambda"), _f32(h0, (B, D), "h0"), _f32(dhT, (B, D), "dhT")
    f32 = dict(dtype=torch.float32, device=x.device)
    out = {"dx": torch.empty_like(x), "dWr": torch.empty((D, D), **f32),
           "dbr": torch.empty(D, **f32), "dWi": torch.empty((D, D), **f32),
           "dbi": torch.empty(D, **f32), "dlambda": torch.empty(D, **f32),
           "dh0": torch.empty((B, D), **f32)}
    ws, nws = _workspace(OP_BACKWARD, B, L, D, io, x.device)
    _check(recblr_bdlru_backward(
        _ptr(x), _ptr(Wr), _ptr(br), _ptr(Wi), _ptr(bi), _ptr(lam), _ptr(h0), _ptr(h), _ptr(dh),
        _ptr(dhT), _ptr(out["dx"]), _ptr(out["dWr"]), _ptr(out["dbr"]), _ptr(out["dWi"]),
        _ptr(out["dbi"]), _ptr(out["dlambda"]), _ptr(out["dh0"]), B, L, D, io, _ptr(ws), nws,
        _stream(stream)), "recblr_bdlru_backward")
    return out


@_on_stream
def bdlru_step(x, Wr, br, Wi, bi, lam, h_prev, out=None, stream=None):
    """Full single step with gate projections; returns h_next (float32)."""
    B, D = x.shape
    io = io_code(x.dtype)
    _f32(lam, (D,), "lambda"), _f32(h_prev, (B, D), "h_prev")
    h_next = torch.empty((B, D), dtype=torch.float32, device=x.device) if out is None else out
    ws, nws = _workspace(OP_STEP, B, 1, D, io, x.device)
    _check(recblr_bdlru_step(_ptr(x), _ptr(Wr), _ptr(br), _ptr(Wi), _ptr(bi), _ptr(lam),
                             _ptr(h_prev), _ptr(h_next), B, D, io, _ptr(ws), nws,
                             _stream(stream)), "recblr_bdlru_step")
    return h_next


@_on_stream
def linear_scan_forward(a, u, h0=None, stream=None):
    """Raw recurrence h_t = a_t h_{t-1} + u_t (float32). Returns (h, hT)."""
    B, L, D = a.shape
    h = torch.empty_like(a)
    hT = torch.empty((B, D), dtype=torch.float32, device=a.device)
    _check(recblr_linear_scan_forward(_ptr(a), _ptr(u), _ptr(h0), _ptr(h), _ptr(hT), B, L, D,
                                      _stream(stream)), "recblr_linear_scan_forward")
    return h, hT


@_on_stream
def scan_backward_method(method, x, zr, zi, lam, h, dh, stream=None):
    """Gated scan backward (zero initial state, no dL/dh_T) by one of SCAN_CHUNKED,
    SCAN_SERIAL, SCAN_TREE. Returns dict dx, dzr, dzi (dtype of x), dlambda (float32)."""
    B, L, D = x.shape
    io = io_code(x.dtype)
    out = {"dx": torch.empty_like(x), "dzr": torch.empty_like(x), "dzi": torch.empty_like(x),
           "dlambda": torch.empty(D, dtype=torch.float32, device=x.device)}
    ws, nws = _workspace(OP_SCAN_BACKWARD_METHOD, B, L, D, io, x.device)
    _check(recblr_scan_backward_method(method, _ptr(x), _ptr(zr), _ptr(zi), _ptr(lam), _ptr(h),
                                       _ptr(dh), _ptr(out["dx"]), _ptr(out["dzr"]),
                                       _ptr(out["dzi"]), _ptr(out["dlambda"]), B, L, D, io,
                                       _ptr(ws), nws, _stream(stream)),
           "recblr_scan_backward_method")
    return out


@_on_stream
def scan_forward_method(method, x, zr, zi, lam, stream=None):
    """Gated scan forward (zero initial state) by one of SCAN_CHUNKED, SCAN_SERIAL,
    SCAN_TREE (the efficiency-ablation variants). Returns h."""
    B, L, D = x.shape
    io = io_code(x.dtype)
    h = torch.empty_like(x)
    ws, nws = _workspace(OP_SCAN_FORWARD, B, L, D, io, x.device)
    _check(recblr_scan_forward_method(method, _ptr(x), _ptr(zr), _ptr(zi), _ptr(lam), _ptr(h),
                                      B, L, D, io, _ptr(ws), nws, _stream(stream)),
           "recblr_scan_forward_method")
    return h


@_on_stream
def gated_forward(hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam, h0=None, keep_h=True,
                  stream=None):
    """Gated recurrent layer core: y = BD-LRU(SiLU(conv(hx))) * SiLU(hz).
    conv_w is [D][K] float32. Returns (y, h, hT) (h is None unless keep_h)."""
    B, L, D = hx.shape
    K = conv_w.shape[1]
    io = io_code(hx.dtype)
    y = torch.empty_like(hx)
    h = torch.empty_like(hx) if keep_h else None
    hT = torch.empty((B, D), dtype=torch.float32, device=hx.device)
    ws, nws = _workspace(OP_GATED_FORWARD, B, L, D, io, hx.device)
    _check(recblr_gated_forward(_ptr(hx), _ptr(hz), _ptr(conv_w), _ptr(conv_b), K, _ptr(Wr),
                                _ptr(br), _ptr(Wi), _ptr(bi), _ptr(lam), _ptr(h0), _ptr(y),
                                _ptr(h), _ptr(hT), B, L, D, io, _ptr(ws), nws, _stream(stream)),
           "recblr_gated_forward")
    return y, h, hT


@_on_stream
def gated_backward(hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam, h, dy, h0=None, dhT=None,
                   stream=None):
    """Backward of gated_forward (h: its BD-LRU output).  Returns a dict with dhx,
    dhz, dconv_w [D][K], dconv_b (None without a conv bias), dWr, dbr, dWi, dbi,
    dlambda, dh0 (None without h0)."""
    B, L, D = hx.shape
    K = conv_w.shape[1]
    io = io_code(hx.dtype)
    f32 = dict(dtype=torch.float32, device=hx.device)
    out = {"dhx": torch.empty_like(hx), "dhz": torch.empty_like(hx),
           "dconv_w": torch.empty((D, K), **f32),
           "dconv_b": torch.empty(D, **f32) if conv_b is not None else None,
           "dWr": torch.empty((D, D), **f32), "dbr": torch.empty(D, **f32),
           "dWi": torch.empty((D, D), **f32), "dbi": torch.empty(D, **f32),
           "dlambda": torch.empty(D, **f32),
           "dh0": torch.empty((B, D), **f32) if h0 is not None else None}
    ws, nws = _workspace(OP_GATED_BACKWARD, B, L, D, io, hx.device)
    _check(recblr_gated_backward(
        _ptr(hx), _ptr(hz), _ptr(conv_w), _ptr(conv_b), K, _ptr(Wr), _ptr(br), _ptr(Wi),
        _ptr(bi), _ptr(lam), _ptr(h0), _ptr(h), _ptr(dy), _ptr(dhT), _ptr(out["dhx"]),
        _ptr(out["dhz"]), _ptr(out["dconv_w"]), _ptr(out["dconv_b"]), _ptr(out["dWr"]),
        _ptr(out["dbr"]), _ptr(out["dWi"]), _ptr(out["dbi"]), _ptr(out["dlambda"]),
        _ptr(out["dh0"]), B, L, D, io, _ptr(ws), nws, _stream(stream)), "recblr_gated_backward")
    return out


# ------------------------------------------------------------------ full model step

def model_dims(B, T, D, E=2, V=3416, layers=2, K=4, eps=1e-12) -> ModelDims:
    return ModelDims(B, T, D, E, V, layers, K, eps)


def model_param_offsets(dims: ModelDims):
    """Offsets (floats) of the flat parameter tensors, in the documented order."""
    n = recblr_model_param_offsets(ctypes.byref(dims), None, 0)
    if n < 0:
        raise RecblrError(ERR_UNSUPPORTED, "recblr_model_param_offsets")
    arr = (ctypes.c_int64 * n)()
    recblr_model_param_offsets(ctypes.byref(dims), arr, n)
    return list(arr)


class ModelStep:
    """One training step of the full model on the GPU: holds the rocBLAS handle
    and the workspace for fixed dimensions."""

    def __init__(self, dims: ModelDims, device="cuda"):
        self.dims = dims
        self.count = recblr_model_param_count(ctypes.byref(dims))
        if self.count == 0:
            raise RecblrError(ERR_UNSUPPORTED, "recblr_model_param_count")
        n = recblr_model_workspace_size(ctypes.byref(dims))
        if n == 0:
            raise RecblrError(ERR_UNSUPPORTED, "recblr_model_workspace_size")
        self.ws = torch.empty(n, dtype=torch.uint8, device=device)
        h = _p()
        _check(recblr_blas_create(ctypes.byref(h)), "recblr_blas_create")
        self.blas = h

    def close(self):
        if self.blas is not None:
            recblr_blas_destroy(self.blas)
            self.blas = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @_on_stream
    def train_step(self, params, ids, targets, grads=None, loss=None, dropout=0.0, seed=0,
                   offset=0, pad_id=-1, stream=None):
        """Loss and gradients (flat, the parameter layout) of one batch; dropout
        with drop probability `dropout` and Philox key (seed, offset), left
        padding with id pad_id (-1: none)."""
        if grads is None:
            grads = torch.empty_like(params)
        if loss is None:
            loss = torch.empty(1, dtype=torch.float32, device=params.device)
        opts = ModelStepOpts(dropout, pad_id, seed, offset)
        _check(recblr_model_train_step(ctypes.byref(self.dims), ctypes.byref(opts), _ptr(params),
                                       _ptr(ids), _ptr(targets), _ptr(grads), _ptr(loss),
                                       _ptr(self.ws), self.ws.numel(), self.blas,
                                       _stream(stream)),
               "recblr_model_train_step")
        return loss, grads


@_on_stream
def adam_update(params, grads, m1, m2, step, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                stream=None):
    _check(recblr_adam_update(_ptr(params), _ptr(grads), _ptr(m1), _ptr(m2), params.numel(),
                              step, lr, beta1, beta2, eps, _stream(stream)), "recblr_adam_update")

