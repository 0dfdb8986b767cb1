"""fp64 CPU oracle of one training step of the full RecBLR model (f4).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The HIP library never imports, links
or calls anything here, and nothing here imports the HIP library.

What it computes, in plain PyTorch CPU ops in float64 (autograd gives the
gradients of the loss; the recurrence is a plain loop over t):

  embedding (section 2, eq:layernorm)   H = LayerNorm(E[ids])
  behaviour-modelling layer, x `layers` (section 3.1):
    gated recurrent layer (Algorithm alg:gated_recurrent)
      Hx = H Wx^T + bx,  Hz = H Wz^T + bz                 (D -> E*D)
      x' = SiLU(b_c + sum_{j<K} w_c[:, j] Hx_{t-j})        (causal, depthwise)
      BD-LRU (section 3.2): z = x' W^T + b, r = sigma(z_r), i = sigma(z_i),
        alpha = exp(-softplus(Lambda) r), beta = sqrt(1 - alpha^2) i,
        h_t = alpha_t h_{t-1} + beta_t x'_t, h_0 = 0
      O = (h (x) SiLU(Hz)) Wo^T + bo                       (E*D -> D)
    H1 = LayerNorm(H + O)
    PFFN (eq. PFFN): Q = SiLU(H1 W1^T + b1) W2^T + b2     (D -> 4D -> D)
    H  = LayerNorm(H1 + Q)
  prediction (section 2): logits = h_T E^T with h_T = H[:, T-1];
  loss = mean over the batch of the cross entropy of softmax(logits) with
  the target item.

Readings of the paper taken here (it leaves them open):
  - the residual connections and layer normalisations sit after each of the
    two sub-layers (post-norm: LayerNorm(x + sublayer(x)));
  - dropout is the identity (evaluation mode; the harness draws no masks);
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
    """Algorithm alg:gated_recurrent, lines 3 to 5, with h_0 = 0 (torch tensors)."""
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


def loss_fn(p, ids, targets, D, E, V, layers, K, eps):
    """Loss of one batch; p maps names to float64 tensors."""
    H = _ln(p["emb"][ids], p["emb_ln_g"], p["emb_ln_b"], eps)
    for l in range(layers):
        g = lambda n: p[f"l{l}.{n}"]
        hx = H @ g("Wx").T + g("bx")
        hz = H @ g("Wz").T + g("bz")
        y = gated_core(hx, hz, g("conv_w"), g("conv_b"), g("Wr"), g("br"), g("Wi"), g("bi"),
                       g("lambda"))
        H1 = _ln(H + (y @ g("Wo").T + g("bo")), g("ln1_g"), g("ln1_b"), eps)
        Q = _silu(H1 @ g("W1").T + g("b1")) @ g("W2").T + g("b2")
        H = _ln(H1 + Q, g("ln2_g"), g("ln2_b"), eps)
    logits = H[:, -1, :] @ p["emb"].T
    lse = torch.logsumexp(logits, dim=-1)
    return (lse - logits[torch.arange(logits.shape[0]), targets]).mean()


def train_step(params, ids, targets, D, E, V, layers, K, eps=1e-12):
    """Loss and the gradient of every parameter (flat, same layout, zero padding).
    params: flat float array; ids: [B][T] ints in [0, V); targets: [B] ints."""
    flat = torch.tensor(np.asarray(params, dtype=np.float64), requires_grad=True)
    p = unflatten(flat, D, E, V, layers, K)
    loss = loss_fn(p, torch.as_tensor(np.asarray(ids, dtype=np.int64)),
                   torch.as_tensor(np.asarray(targets, dtype=np.int64)), D, E, V, layers, K, eps)
    loss.backward()
    return float(loss.detach()), flat.grad.numpy().copy()


def adam(params, grads, m1, m2, step, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8):
    """One Adam update (Kingma and Ba, Algorithm 1), in place on float64 arrays."""
    m1[:] = beta1 * m1 + (1.0 - beta1) * grads
    m2[:] = beta2 * m2 + (1.0 - beta2) * grads * grads
    mhat = m1 / (1.0 - beta1 ** step)
    vhat = m2 / (1.0 - beta2 ** step)
    params[:] = params - lr * mhat / (np.sqrt(vhat) + eps)
