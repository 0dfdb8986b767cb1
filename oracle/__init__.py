"""fp64 CPU oracle of the BD-LRU scan (RecBLR, arXiv 2406.12580, section 3.2).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The HIP library never imports, links
or calls anything here, and nothing here imports the HIP library.

The arithmetic lives in ``recblr_oracle.c`` (a plain sequential loop over t
per channel, in double precision); this module compiles it with gcc when the
shared object is missing or older than its source and wraps it with ctypes.
Every function takes numpy arrays of any real dtype, widens them exactly to
float64 and returns float64 arrays.  ``oracle.model`` holds the oracle of a
whole model training step (plain PyTorch CPU ops in float64).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "recblr_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math) and return the .so path."""
    stale = not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)
    if force or stale:
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                        "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        i64, p = ctypes.c_int64, ctypes.c_void_p
        sigs = {
            "oracle_linear_scan": [i64, i64, i64, p, p, p, p, p],
            "oracle_scan_forward": [i64, i64, i64, p, p, p, p, p, p, p],
            "oracle_scan_step": [i64, i64, p, p, p, p, p, p],
            "oracle_scan_backward": [i64, i64, i64] + [p] * 12,
            "oracle_project": [i64, i64, p, p, p, p],
            "oracle_forward": [i64, i64, i64] + [p] * 9,
            "oracle_backward": [i64, i64, i64] + [p] * 16,
            "oracle_step": [i64, i64] + [p] * 8,
            "oracle_gated_forward": [i64, i64, i64, i64] + [p] * 13,
            "oracle_gated_backward": [i64, i64, i64, i64] + [p] * 22,
        }
        for name, args in sigs.items():
            fn = getattr(_lib, name)
            fn.argtypes = args
            fn.restype = None
    return _lib


def _in(a):
    """Widen an input to a C-contiguous float64 array (exact for fp32 and bf16 values)."""
    return None if a is None else np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data


def linear_scan(a, u, h0=None):
    """h_t = a_t h_{t-1} + u_t over [B, L, D]; returns (h, hT)."""
    a, u, h0 = _in(a), _in(u), _in(h0)
    B, L, D = a.shape
    h = np.empty_like(a)
    hT = np.empty((B, D))
    _load().oracle_linear_scan(B, L, D, _ptr(a), _ptr(u), _ptr(h0), _ptr(h), _ptr(hT))
    return h, hT


def scan_forward(x, zr, zi, lam, h0=None):
    """Gated BD-LRU scan from pre-activations; returns (h [B,L,D], hT [B,D])."""
    x, zr, zi, lam, h0 = map(_in, (x, zr, zi, lam, h0))
    B, L, D = x.shape
    h = np.empty_like(x)
    hT = np.empty((B, D))
    _load().oracle_scan_forward(B, L, D, _ptr(x), _ptr(zr), _ptr(zi), _ptr(lam), _ptr(h0),
                                _ptr(h), _ptr(hT))
    return h, hT


def scan_step(x, zr, zi, lam, h_prev):
    """One recurrent step over [B, D]; returns h_next."""
    x, zr, zi, lam, h_prev = map(_in, (x, zr, zi, lam, h_prev))
    B, D = x.shape
    out = np.empty_like(x)
    _load().oracle_scan_step(B, D, _ptr(x), _ptr(zr), _ptr(zi), _ptr(lam), _ptr(h_prev),
                             _ptr(out))
    return out


def scan_backward(x, zr, zi, lam, dh, h0=None, dhT=None):
    """Adjoint of scan_forward; returns dict dx, dzr, dzi, dlambda, dh0."""
    x, zr, zi, lam, dh, h0, dhT = map(_in, (x, zr, zi, lam, dh, h0, dhT))
    B, L, D = x.shape
    out = {k: np.empty_like(x) for k in ("dx", "dzr", "dzi")}
    out["dlambda"] = np.empty(D)
    out["dh0"] = np.empty((B, D))
    _load().oracle_scan_backward(B, L, D, _ptr(x), _ptr(zr), _ptr(zi), _ptr(lam), _ptr(h0),
                                 _ptr(dh), _ptr(dhT), _ptr(out["dx"]), _ptr(out["dzr"]),
                                 _ptr(out["dzi"]), _ptr(out["dlambda"]), _ptr(out["dh0"]))
    return out


def project(x, W, b=None):
    """z = x W^T + b over the last axis of x (W is [out, in])."""
    x, W, b = _in(x), _in(W), _in(b)
    D = x.shape[-1]
    M = x.size // D if D else 0
    z = np.empty(x.shape[:-1] + (W.shape[0],))
    _load().oracle_project(M, D, _ptr(x), _ptr(W), _ptr(b), _ptr(z))
    return z


def forward(x, Wr, br, Wi, bi, lam, h0=None):
    """Full BD-LRU forward with gate projections; returns (h, hT)."""
    x, Wr, br, Wi, bi, lam, h0 = map(_in, (x, Wr, br, Wi, bi, lam, h0))
    B, L, D = x.shape
    h = np.empty_like(x)
    hT = np.empty((B, D))
    _load().oracle_forward(B, L, D, _ptr(x), _ptr(Wr), _ptr(br), _ptr(Wi), _ptr(bi), _ptr(lam),
                           _ptr(h0), _ptr(h), _ptr(hT))
    return h, hT


def backward(x, Wr, br, Wi, bi, lam, dh, h0=None, dhT=None):
    """Full BD-LRU backward; returns dict dx, dWr, dbr, dWi, dbi, dlambda, dh0."""
    x, Wr, br, Wi, bi, lam, dh, h0, dhT = map(_in, (x, Wr, br, Wi, bi, lam, dh, h0, dhT))
    B, L, D = x.shape
    out = {"dx": np.empty_like(x), "dWr": np.empty((D, D)), "dbr": np.empty(D),
           "dWi": np.empty((D, D)), "dbi": np.empty(D), "dlambda": np.empty(D),
           "dh0": np.empty((B, D))}
    _load().oracle_backward(B, L, D, _ptr(x), _ptr(Wr), _ptr(br), _ptr(Wi), _ptr(bi), _ptr(lam),
                            _ptr(h0), _ptr(dh), _ptr(dhT), _ptr(out["dx"]), _ptr(out["dWr"]),
                            _ptr(out["dbr"]), _ptr(out["dWi"]), _ptr(out["dbi"]),
                            _ptr(out["dlambda"]), _ptr(out["dh0"]))
    return out


def step(x, Wr, br, Wi, bi, lam, h_prev):
    """Full single step with gate projections; returns h_next [B, D]."""
    x, Wr, br, Wi, bi, lam, h_prev = map(_in, (x, Wr, br, Wi, bi, lam, h_prev))
    B, D = x.shape
    out = np.empty_like(x)
    _load().oracle_step(B, D, _ptr(x), _ptr(Wr), _ptr(br), _ptr(Wi), _ptr(bi), _ptr(lam),
                        _ptr(h_prev), _ptr(out))
    return out


def gated_forward(hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam, h0=None):
    """Gated recurrent layer core (Algorithm alg:gated_recurrent):
    x' = SiLU(causal depthwise Conv1d(hx)), h = BD-LRU(x'), y = h * SiLU(hz).
    conv_w is [D][K]. Returns (y, h, hT)."""
    hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam, h0 = map(
        _in, (hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam, h0))
    B, L, D = hx.shape
    K = conv_w.shape[1]
    y = np.empty_like(hx)
    h = np.empty_like(hx)
    hT = np.empty((B, D))
    _load().oracle_gated_forward(B, L, D, K, _ptr(hx), _ptr(hz), _ptr(conv_w), _ptr(conv_b),
                                 _ptr(Wr), _ptr(br), _ptr(Wi), _ptr(bi), _ptr(lam), _ptr(h0),
                                 _ptr(y), _ptr(h), _ptr(hT))
    return y, h, hT


def gated_backward(hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam, dy, h0=None, dhT=None):
    """Backward of gated_forward (exact adjoint).  Returns a dict with dhx, dhz,
    dconv_w [D][K], dconv_b [D], dWr, dbr, dWi, dbi, dlambda, dh0."""
    hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam, dy, h0, dhT = map(
        _in, (hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam, dy, h0, dhT))
    B, L, D = hx.shape
    K = conv_w.shape[1]
    out = {"dhx": np.empty_like(hx), "dhz": np.empty_like(hx), "dconv_w": np.empty((D, K)),
           "dconv_b": np.empty(D), "dWr": np.empty((D, D)), "dbr": np.empty(D),
           "dWi": np.empty((D, D)), "dbi": np.empty(D), "dlambda": np.empty(D),
           "dh0": np.empty((B, D))}
    _load().oracle_gated_backward(
        B, L, D, K, _ptr(hx), _ptr(hz), _ptr(conv_w), _ptr(conv_b), _ptr(Wr), _ptr(br),
        _ptr(Wi), _ptr(bi), _ptr(lam), _ptr(h0), _ptr(dy), _ptr(dhT), _ptr(out["dhx"]),
        _ptr(out["dhz"]), _ptr(out["dconv_w"]), _ptr(out["dconv_b"]), _ptr(out["dWr"]),
        _ptr(out["dbr"]), _ptr(out["dWi"]), _ptr(out["dbi"]), _ptr(out["dlambda"]),
        _ptr(out["dh0"]))
    return out
