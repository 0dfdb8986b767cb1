"""fp64 CPU oracle of one training step of the full RecBLR model (f4).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The HIP library never imports, links
or calls anything here, and nothing here imports the HIP library.

What it computes, in plain PyTorch CPU ops in float64 (autograd gives the
gradients of the loss; the recurrence is a plain loop over t):

  embedding (section 2, eq:layernorm)   H = LayerNorm(Dropout(E[ids]))
    (a position holding the padding id takes the zero vector instead of a
    row of E: left padding with zeros, section 3.3)
  behaviour-modelling layer, x `layers` (section 3.1):
    gated recurrent layer (Algorithm alg:gated_recurrent)
      Hx = H Wx^T + bx,  Hz = H Wz^T + bz                 (D -> E*D)
      x' = SiLU(b_c + sum_{j<K} w_c[:, j] Hx_{t-j})        (causal, depthwise)
      BD-LRU (section 3.2): z = x' W^T + b, r = sigma(z_r), i = sigma(z_i),
        alpha = exp(-softplus(Lambda) r), beta = sqrt(1 - alpha^2) i,
        h_t = alpha_t h_{t-1} + beta_t x'_t, h_0 = 0
      O = (h (x) SiLU(Hz)) Wo^T + bo                       (E*D -> D)
    H1 = LayerNorm(H + Dropout(O))
    PFFN (eq. PFFN): Q = SiLU(H1 W1^T + b1) W2^T + b2     (D -> 4D -> D)
    H  = LayerNorm(H1 + Dropout(Q))
  prediction (section 2): logits = h_T E^T with h_T = H[:, T-1];
  loss = mean over the batch of the cross entropy of softmax(logits) with
  the target item.

Readings of the paper taken here (it leaves them open):
  - the residual connections and layer normalisations sit after each of the
    two sub-layers (post-norm: LayerNorm(x + sublayer(x)));
  - dropout (section 3.1 names it beside the residuals and layer norms
    without placing it) sits on the embedding and on each sub-layer's output
    before its residual sum; it is inverted dropout: an element is kept with
    probability 1 - p and then scaled by 1 / (1 - p).  Its masks come from a
    counter-based generator, Philox4x64-10, so that any implementation can
    draw the same ones: element e (row-major over [B][T][D]) of dropout site
    s (0 the embedding, 1 + 2l layer l's gated recurrent output, 2 + 2l its
    PFFN output) takes 32-bit word e mod 8 (low half of each 64-bit output
    word first) of Philox4x64-10 at counter (floor(e / 8), s, 0, 0) and key
    (seed, offset); it is dropped when that word is below floor(p 2^32), p
    taken as a float32;
  - the padding id marks left padding: such a position enters the model as
    the zero vector (the lookup sends no gradient to E there) and is
    otherwise processed like any other position; the softmax runs over all V
    ids;
  - the LayerNorm epsilon is a parameter (`eps`), the conv has K taps and a
    bias per channel, the BD-LRU starts from a zero state;
  - the loss is the cross entropy of the next item at the last position.

Parameters live in one flat float vector; `layout` gives the order (the
order documented with the C ABI's model entry points), each tensor starting
at a multiple of 64 floats.  Weights are [out][in].
"""
from __future__ import annotations

import numpy as np
import torch

ALIGN = 64


# Philox4x64-10: Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
# easy as 1, 2, 3" (SC 2011).  Ten rounds over a 4 x 64-bit counter; each
# round multiplies counter words 0 and 2 by the two round multipliers, and
# the output is (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1,
# lo(M0 c0)); the key words are bumped by the two Weyl constants between
# rounds.
PHILOX_M = (0xD2E7470EE14C6C93, 0xCA5A826395121157)
PHILOX_W = (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)
_LO32 = np.uint64(0xFFFFFFFF)


def _mulhilo64(a, b):
    """Low and high 64 bits of the 128-bit products a * b (uint64 arrays),
    from the four 32 x 32-bit partial products."""
    s32 = np.uint64(32)
    a0, a1, b0, b1 = a & _LO32, a >> s32, b & _LO32, b >> s32
    p00, p01, p10, p11 = a0 * b0, a0 * b1, a1 * b0, a1 * b1
    mid = (p00 >> s32) + (p01 & _LO32) + (p10 & _LO32)
    return a * b, p11 + (p01 >> s32) + (p10 >> s32) + (mid >> s32)


def philox4x64_10(c0, c1, c2, c3, k0, k1):
    """Philox4x64-10 of the counters (c0, c1, c2, c3) under key (k0, k1):
    four uint64 arrays (the arguments broadcast)."""
    u = lambda v: np.asarray(v, dtype=np.uint64)
    c = np.broadcast_arrays(u(c0), u(c1), u(c2), u(c3))
    c = [x.copy() for x in c]
    k = [u(k0), u(k1)]
    m0, m1 = u(PHILOX_M[0]), u(PHILOX_M[1])
    with np.errstate(over="ignore"):
        for r in range(10):
            if r:
                k = [k[0] + u(PHILOX_W[0]), k[1] + u(PHILOX_W[1])]
            lo0, hi0 = _mulhilo64(m0, c[0])
            lo1, hi1 = _mulhilo64(m1, c[2])
            c = [hi1 ^ c[1] ^ k[0], lo1, hi0 ^ c[3] ^ k[1], lo0]
    return c


def drop_threshold(p) -> int:
    """floor(p 2^32) for p taken as a float32: a 32-bit word below it drops."""
    return int(np.floor(np.float64(np.float32(p)) * 2.0 ** 32))


def dropout_keep(site: int, n: int, p, seed: int, offset: int):
    """Keep flags (bool [n]) of elements 0 .. n-1 of dropout site `site`."""
    g = np.arange((n + 7) // 8, dtype=np.uint64)
    words = np.stack(philox4x64_10(g, site, 0, 0, seed, offset), axis=1)  # [G][4]
    u32 = np.stack([words & _LO32, words >> np.uint64(32)], axis=2).reshape(-1)[:n]
    return u32 >= np.uint64(drop_threshold(p))


def layer_tensors(D: int, E: int, K: int):
    ED = E * D
    return [("Wx", (ED, D)), ("bx", (ED,)), ("Wz", (ED, D)), ("bz", (ED,)),
            ("conv_w", (ED, K)), ("conv_b", (ED,)), ("Wr", (ED, ED)), ("br", (ED,)),
            ("Wi", (ED, ED)), ("bi", (ED,)), ("lambda", (ED,)), ("Wo", (D, ED)), ("bo", (D,)),
            ("ln1_g", (D,)), ("ln1_b", (D,)), ("W1", (4 * D, D)), ("b1", (4 * D,)),
            ("W2", (D, 4 * D)), ("b2", (D,)), ("ln2_g", (D,)), ("ln2_b", (D,))]


def layout(D: int, E: int, V: int, layers: int, K: int):
    """[(name, shape, offset)], total: the flat parameter order."""
    items = [("emb", (V, D)), ("emb_ln_g", (D,)), ("emb_ln_b", (D,))]
    for l in range(layers):
        items += [(f"l{l}.{n}", s) for n, s in layer_tensors(D, E, K)]
    out, off = [], 0
    for name, shape in items:
        out.append((name, shape, off))
        off += -(-int(np.prod(shape)) // ALIGN) * ALIGN
    return out, off


def unflatten(flat, D, E, V, layers, K):
    lay, _ = layout(D, E, V, layers, K)
    return {n: flat[o:o + int(np.prod(s))].reshape(s) for n, s, o in lay}


def _ln(x, g, b, eps):
    mu = x.mean(dim=-1, keepdim=True)
    var = ((x - mu) ** 2).mean(dim=-1, keepdim=True)
    return (x - mu) / torch.sqrt(var + eps) * g + b


def _silu(v):
    return v * torch.sigmoid(v)


def _softplus(v):
    return torch.clamp(v, min=0.0) + torch.log1p(torch.exp(-torch.abs(v)))


def gated_core(hx, hz, conv_w, conv_b, Wr, br, Wi, bi, lam):
    """The core of Algorithm alg:gated_recurrent (causal conv + SiLU, BD-LRU,
    output gate), with h_0 = 0 (torch tensors)."""
    B, T, C = hx.shape
    K = conv_w.shape[1]
    c = conv_b.expand(B, T, C).clone()
    for j in range(K):
        if j < T:
            c[:, j:, :] = c[:, j:, :] + conv_w[:, j] * hx[:, :T - j, :]
    xp = _silu(c)
    r = torch.sigmoid(xp @ Wr.T + br)
    i = torch.sigmoid(xp @ Wi.T + bi)
    q = _softplus(lam) * r
    alpha = torch.exp(-q)
    beta = torch.sqrt(-torch.expm1(-2.0 * q)) * i
    h = torch.zeros(B, C, dtype=hx.dtype)
    outs = []
    for t in range(T):
        h = alpha[:, t] * h + beta[:, t] * xp[:, t]
        outs.append(h)
    H = torch.stack(outs, dim=1) if T > 0 else torch.zeros(B, 0, C, dtype=hx.dtype)
    return H * _silu(hz)


def hidden(p, ids, D, E, V, layers, K, eps, dropout=0.0, seed=0, offset=0, pad_id=-1):
    """Output H [B][T][D] of the last behaviour-modelling layer; p maps names
    to float64 tensors.  dropout: drop probability in [0, 1); seed, offset:
    the Philox key; pad_id: the padding id (-1: none)."""
    def drop(x, site):
        if dropout == 0.0:
            return x
        keep = dropout_keep(site, x.numel(), dropout, seed, offset).reshape(tuple(x.shape))
        return x * torch.as_tensor(keep, dtype=x.dtype) / (1.0 - float(np.float32(dropout)))

    X0 = p["emb"][ids]
    if pad_id >= 0:
        X0 = X0 * (ids != pad_id).unsqueeze(-1).to(X0.dtype)
    H = _ln(drop(X0, 0), p["emb_ln_g"], p["emb_ln_b"], eps)
    for l in range(layers):
        g = lambda n: p[f"l{l}.{n}"]
        hx = H @ g("Wx").T + g("bx")
        hz = H @ g("Wz").T + g("bz")
        y = gated_core(hx, hz, g("conv_w"), g("conv_b"), g("Wr"), g("br"), g("Wi"), g("bi"),
                       g("lambda"))
        H1 = _ln(H + drop(y @ g("Wo").T + g("bo"), 1 + 2 * l), g("ln1_g"), g("ln1_b"), eps)
        Q = _silu(H1 @ g("W1").T + g("b1")) @ g("W2").T + g("b2")
        H = _ln(H1 + drop(Q, 2 + 2 * l), g("ln2_g"), g("ln2_b"), eps)
    return H


def loss_fn(p, ids, targets, D, E, V, layers, K, eps, dropout=0.0, seed=0, offset=0,
            pad_id=-1):
    """Loss of one batch (arguments as for hidden)."""
    H = hidden(p, ids, D, E, V, layers, K, eps, dropout, seed, offset, pad_id)
    logits = H[:, -1, :] @ p["emb"].T
    lse = torch.logsumexp(logits, dim=-1)
    return (lse - logits[torch.arange(logits.shape[0]), targets]).mean()


def train_step(params, ids, targets, D, E, V, layers, K, eps=1e-12, dropout=0.0, seed=0,
               offset=0, pad_id=-1):
    """Loss and the gradient of every parameter (flat, same layout, zero padding).
    params: flat float array; ids: [B][T] ints in [0, V); targets: [B] ints;
    dropout, seed, offset, pad_id as for loss_fn."""
    flat = torch.tensor(np.asarray(params, dtype=np.float64), requires_grad=True)
    p = unflatten(flat, D, E, V, layers, K)
    loss = loss_fn(p, torch.as_tensor(np.asarray(ids, dtype=np.int64)),
                   torch.as_tensor(np.asarray(targets, dtype=np.int64)), D, E, V, layers, K, eps,
                   dropout, seed, offset, pad_id)
    loss.backward()
    return float(loss.detach()), flat.grad.numpy().copy()


def adam(params, grads, m1, m2, step, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8):
    """One Adam update (Kingma and Ba, Algorithm 1), in place on float64 arrays."""
    m1[:] = beta1 * m1 + (1.0 - beta1) * grads
    m2[:] = beta2 * m2 + (1.0 - beta2) * grads * grads
    mhat = m1 / (1.0 - beta1 ** step)
    vhat = m2 / (1.0 - beta2 ** step)
    params[:] = params - lr * mhat / (np.sqrt(vhat) + eps)
