"""Seeded synthetic inputs for the BD-LRU scan.

This module is shared by the parity tests, the benchmark and the smoke check:
it feeds the same numbers to the HIP library and to the fp64 oracle.  It holds
none of the method's arithmetic, only the input recipe:

* x, the gate pre-activations z_r, z_i and the upstream gradient dL/dh are
  standard normal draws.  Drawing z directly stands in for W x with
  W ~ N(0, 1/D) and x ~ N(0, 1), whose entries have unit variance.
* The decay parameter follows the paper's initialisation (section 3.2): a
  per-channel base a_d ~ U[lo, hi] and Lambda_d = ln(1/a_d - 1), so that
  exp(-softplus(Lambda_d)) = a_d.
* For bf16 I/O every tensor the kernel reads in bf16 is rounded to nearest
  even from its fp32 draw; the arrays stay float32 but hold bf16 values.

Every generator draws from numpy's PCG64 with an explicit seed.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    rounded = ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16) << 16
    nan = np.isnan(a)
    out = rounded.astype(np.uint32).view(np.float32).copy()
    out[nan] = np.float32("nan")
    return out


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bf16-representable."""
    return (np.ascontiguousarray(a, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def bf16_from_bits(bits: np.ndarray) -> np.ndarray:
    """Widen raw bfloat16 bit patterns to float32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def lambda_from_base(a: np.ndarray) -> np.ndarray:
    """Lambda such that exp(-softplus(Lambda)) equals the decay base a (0 < a < 1)."""
    a = np.asarray(a, dtype=np.float64)
    return np.log(1.0 / a - 1.0).astype(np.float32)


@dataclass
class Config:
    name: str
    B: int
    L: int
    D: int
    io: str            # "f32" or "bf16": the dtype of x, z and h in HBM
    a_range: tuple     # per-channel decay base range
    seed: int
    ops: tuple         # "fwd", "bwd", "step"
    note: str = ""


# The synthetic workloads: typical next-item training batches (D = 64, L = 200,
# batch 2048), long user histories (L = 2048, D = 128) and very long histories
# in bf16 (L = 16384, D = 256) plus a one-step decode over 65536 users.
CONFIGS = {
    "c1": Config("c1", 4, 50, 64, "f32", (0.9, 0.999), 1, ("fwd",), "small case"),
    "c2": Config("c2", 256, 200, 64, "f32", (0.9, 0.999), 2, ("fwd",), "training batch"),
    "c3": Config("c3", 2048, 200, 64, "f32", (0.9, 0.999), 3, ("fwd", "bwd"), "batch 2048"),
    "c4": Config("c4", 256, 2048, 128, "f32", (0.99, 0.9999), 4, ("fwd", "bwd"),
                 "long histories"),
    "c5": Config("c5", 16, 16384, 256, "bf16", (0.99, 0.9999), 5, ("fwd", "bwd"),
                 "very long histories, bf16 I/O"),
    "c5dec": Config("c5dec", 65536, 1, 256, "bf16", (0.99, 0.9999), 6, ("step",),
                    "single-step decode"),
}


@dataclass
class ScanInputs:
    x: np.ndarray
    zr: np.ndarray
    zi: np.ndarray
    lam: np.ndarray
    h0: np.ndarray | None = None
    dh: np.ndarray | None = None
    dhT: np.ndarray | None = None
    io: str = "f32"
    extra: dict = field(default_factory=dict)


def _normal(rng, shape, io):
    a = rng.standard_normal(shape, dtype=np.float32)
    return round_bf16(a) if io == "bf16" else a


def scan_inputs(B, L, D, seed, io="f32", a_range=(0.9, 0.999), h0=False, grad=False,
                dhT=False, silu_x=False, pad_rows=False) -> ScanInputs:
    """Inputs of the scan-level entry points (pre-activations given).

    h0: draw the initial state from N(0, 1) (fp32), else None (zero state).
    grad: also draw dL/dh ~ N(0, 1) in the I/O dtype.
    dhT: also draw dL/dh_T ~ N(0, 1) (fp32).
    silu_x: pass x through SiLU, as the BD-LRU input comes out of a SiLU.
    pad_rows: left-pad every row with zeros to a random valid length in [1, L].
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal((B, L, D), dtype=np.float32)
    if silu_x:
        x = (x / (1.0 + np.exp(-x.astype(np.float64)))).astype(np.float32)
    lengths = None
    if pad_rows:
        lengths = rng.integers(1, L + 1, size=B) if L > 0 else np.zeros(B, dtype=np.int64)
        for b in range(B):
            x[b, : L - lengths[b]] = 0.0
    if io == "bf16":
        x = round_bf16(x)
    zr = _normal(rng, (B, L, D), io)
    zi = _normal(rng, (B, L, D), io)
    lam = lambda_from_base(rng.uniform(a_range[0], a_range[1], size=D))
    out = ScanInputs(x, zr, zi, lam, io=io)
    if h0:
        out.h0 = rng.standard_normal((B, D), dtype=np.float32)
    if grad:
        out.dh = _normal(rng, (B, L, D), io)
    if dhT:
        out.dhT = rng.standard_normal((B, D), dtype=np.float32)
    if lengths is not None:
        out.extra["lengths"] = lengths
    return out


def config_inputs(cfg: Config, grad=None) -> ScanInputs:
    """Inputs of a named workload at its full size (h0 = 0, as the workload states)."""
    want_grad = ("bwd" in cfg.ops) if grad is None else grad
    return scan_inputs(cfg.B, cfg.L, cfg.D, cfg.seed, cfg.io, cfg.a_range, grad=want_grad)


@dataclass
class FullInputs:
    x: np.ndarray
    Wr: np.ndarray
    br: np.ndarray
    Wi: np.ndarray
    bi: np.ndarray
    lam: np.ndarray
    h0: np.ndarray | None = None
    dh: np.ndarray | None = None
    dhT: np.ndarray | None = None
    io: str = "f32"


def full_inputs(B, L, D, seed, io="f32", a_range=(0.9, 0.999), bias=False, h0=False,
                grad=False, dhT=False) -> FullInputs:
    """Inputs of the entry points that take gate parameters: W ~ N(0, 1/D), b = 0 or U[-1, 1]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = _normal(rng, (B, L, D), io)
    scale = np.float32(1.0 / np.sqrt(D)) if D > 0 else np.float32(1.0)
    Wr = rng.standard_normal((D, D), dtype=np.float32) * scale
    Wi = rng.standard_normal((D, D), dtype=np.float32) * scale
    if io == "bf16":
        Wr, Wi = round_bf16(Wr), round_bf16(Wi)
    if bias:
        br = rng.uniform(-1.0, 1.0, size=D).astype(np.float32)
        bi = rng.uniform(-1.0, 1.0, size=D).astype(np.float32)
    else:
        br = np.zeros(D, np.float32)
        bi = np.zeros(D, np.float32)
    if io == "bf16":
        br, bi = round_bf16(br), round_bf16(bi)
    lam = lambda_from_base(rng.uniform(a_range[0], a_range[1], size=D))
    out = FullInputs(x, Wr, br, Wi, bi, lam, io=io)
    if h0:
        out.h0 = rng.standard_normal((B, D), dtype=np.float32)
    if grad:
        out.dh = _normal(rng, (B, L, D), io)
    if dhT:
        out.dhT = rng.standard_normal((B, D), dtype=np.float32)
    return out


def step_inputs(B, D, seed, io="bf16", a_range=(0.99, 0.9999)):
    """Inputs of one recurrent step: x_t, z_r, z_i in the I/O dtype, h_prev ~ N(0, 1) fp32."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = _normal(rng, (B, D), io)
    zr = _normal(rng, (B, D), io)
    zi = _normal(rng, (B, D), io)
    lam = lambda_from_base(rng.uniform(a_range[0], a_range[1], size=D))
    h_prev = rng.standard_normal((B, D), dtype=np.float32)
    return ScanInputs(x, zr, zi, lam, h0=h_prev, io=io)


# ------------------------------------------------------------------ full model (f4)
@dataclass
class ModelDims:
    B: int
    T: int
    D: int
    E: int = 2          # expansion factor of the gated recurrent layer
    V: int = 3416       # items (MovieLens-1M after the paper's preprocessing)
    layers: int = 2     # behaviour-modelling layers (section 4 implementation details)
    K: int = 4          # conv taps
    eps: float = 1e-12  # LayerNorm epsilon


# MovieLens-1M training shape of the paper's implementation details: batch
# 2048, maximum length 200, embedding dimension 64, expansion factor 2, two
# behaviour-modelling layers, 3,416 items.
MODEL_CONFIGS = {
    "ml1m": ModelDims(B=2048, T=200, D=64),
    "ml1m-small": ModelDims(B=4, T=37, D=64, V=211),
}


def model_params(dims: ModelDims, seed: int) -> dict:
    """Named float32 parameters, in the flat parameter order of the model step
    (embedding, its LayerNorm, then each layer's tensors): weights ~ N(0, 1/fan_in),
    biases ~ U[-0.1, 0.1],
    embeddings ~ N(0, 1), LayerNorm gains 1 + U[-0.1, 0.1] and shifts U[-0.1, 0.1],
    conv taps ~ N(0, 1/K), and Lambda from decay bases a ~ U[0.9, 0.999]
    (the paper's initialisation)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    D, E, V, K = dims.D, dims.E, dims.V, dims.K
    ED = E * D
    f32 = lambda a: np.asarray(a, dtype=np.float32)
    w = lambda o, i: f32(rng.standard_normal((o, i)) / np.sqrt(i))
    u = lambda n, s=0.1: f32(rng.uniform(-s, s, n))
    p = {"emb": f32(rng.standard_normal((V, D))), "emb_ln_g": f32(1.0 + u(D)),
         "emb_ln_b": u(D)}
    for l in range(dims.layers):
        q = {"Wx": w(ED, D), "bx": u(ED), "Wz": w(ED, D), "bz": u(ED),
             "conv_w": f32(rng.standard_normal((ED, K)) / np.sqrt(K)), "conv_b": u(ED),
             "Wr": w(ED, ED), "br": u(ED), "Wi": w(ED, ED), "bi": u(ED),
             "lambda": f32(lambda_from_base(rng.uniform(0.9, 0.999, ED))),
             "Wo": w(D, ED), "bo": u(D), "ln1_g": f32(1.0 + u(D)), "ln1_b": u(D),
             "W1": w(4 * D, D), "b1": u(4 * D), "W2": w(D, 4 * D), "b2": u(D),
             "ln2_g": f32(1.0 + u(D)), "ln2_b": u(D)}
        p.update({f"l{l}.{k}": v for k, v in q.items()})
    return p


def model_batch(dims: ModelDims, seed: int, min_len: int | None = None, pad_id: int = 0):
    """Item ids [B][T] and next-item targets [B] (int32), drawn with Zipf(1)
    popularity over the V items (item v has weight 1 / (v + 1)).

    With min_len given, the batch holds short sequences instead: row b has a
    length l_b ~ U{min_len, ..., T}, its first T - l_b positions hold pad_id
    (left padding) and its items and target are drawn, with the same Zipf
    weights, from the V - 1 ids other than pad_id."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if min_len is None:
        pr = 1.0 / np.arange(1, dims.V + 1, dtype=np.float64)
        pr /= pr.sum()
        ids = rng.choice(dims.V, size=(dims.B, dims.T), p=pr).astype(np.int32)
        targets = rng.choice(dims.V, size=dims.B, p=pr).astype(np.int32)
        return ids, targets
    if not 1 <= min_len <= dims.T or not 0 <= pad_id < dims.V:
        raise ValueError("need 1 <= min_len <= T and 0 <= pad_id < V")
    items = np.array([v for v in range(dims.V) if v != pad_id])
    pr = 1.0 / np.arange(1, dims.V, dtype=np.float64)
    pr /= pr.sum()
    lengths = rng.integers(min_len, dims.T, size=dims.B, endpoint=True)
    ids = items[rng.choice(dims.V - 1, size=(dims.B, dims.T), p=pr)].astype(np.int32)
    ids[np.arange(dims.T)[None, :] < (dims.T - lengths)[:, None]] = pad_id
    targets = items[rng.choice(dims.V - 1, size=dims.B, p=pr)].astype(np.int32)
    return ids, targets


def ml1m_min_len(T: int = 200) -> int:
    """Shortest length of the MovieLens-1M length mix: U{m, ..., T} has mean
    (m + T) / 2, so m = 2 * 165.5 - 200 = 131 gives the dataset's average
    length of 165.5 (table tab:dataset) under the maximum length 200; other
    T keep the ratio of mean to maximum length (m = 0.655 T)."""
    return max(1, int(round(T * (2 * 165.5 / 200 - 1))))
