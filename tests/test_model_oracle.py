"""Pins of the fp64 model-step oracle (oracle/model.py): the full RecBLR model
of sections 2 and 3.1 (embedding + LayerNorm, gated recurrent layer, PFFN,
residuals, prediction with softmax cross entropy), and Adam.

Each piece is checked against something other than itself: its gated core
against the C oracle (whose forward and backward are pinned in
test_oracle_pins.py), LayerNorm, PFFN and the loss against closed forms and
numpy written out independently, the residual structure by zeroing
sub-layers, and the whole gradient against central differences.
"""
import numpy as np
import pytest
import torch
from scipy.special import expit, logsumexp

import oracle
from oracle import model as om
from paper_2406_12580_amd import datagen as dg

TINY = dg.ModelDims(B=2, T=5, D=4, E=2, V=7, layers=2, K=3, eps=1e-5)


def _flat(dims, named):
    lay, total = om.layout(dims.D, dims.E, dims.V, dims.layers, dims.K)
    flat = np.zeros(total)
    for n, s, o in lay:
        flat[o:o + int(np.prod(s))] = np.asarray(named[n], dtype=np.float64).ravel()
    return flat


def _setup(dims=TINY, seed=5):
    named = dg.model_params(dims, seed)
    ids, targets = dg.model_batch(dims, seed + 1)
    return named, ids, targets


def _loss(dims, named, ids, targets):
    p = {k: torch.tensor(np.asarray(v, dtype=np.float64)) for k, v in named.items()}
    return float(om.loss_fn(p, torch.as_tensor(ids.astype(np.int64)),
                            torch.as_tensor(targets.astype(np.int64)), dims.D, dims.E, dims.V,
                            dims.layers, dims.K, dims.eps))


def test_layout_is_aligned_and_dense():
    lay, total = om.layout(64, 2, 3416, 2, 4)
    assert [n for n, _, _ in lay][:4] == ["emb", "emb_ln_g", "emb_ln_b", "l0.Wx"]
    end = 0
    for n, s, o in lay:
        assert o % 64 == 0 and o >= end
        end = o + int(np.prod(s))
    assert total == -(-end // 64) * 64
    assert len(lay) == 3 + 2 * 21


def test_gated_core_matches_c_oracle():
    """Values and every gradient of the torch gated core against the C oracle."""
    B, T, C, K = 2, 9, 6, 3
    rng = np.random.default_rng(11)
    hx, hz, dy = (rng.standard_normal((B, T, C)) for _ in range(3))
    w, cb = rng.standard_normal((C, K)), rng.standard_normal(C) * 0.1
    Wr, Wi = rng.standard_normal((C, C)) / np.sqrt(C), rng.standard_normal((C, C)) / np.sqrt(C)
    br, bi = rng.uniform(-1, 1, C), rng.uniform(-1, 1, C)
    lam = np.asarray(dg.lambda_from_base(rng.uniform(0.9, 0.999, C)), dtype=np.float64)
    args = [torch.tensor(a, requires_grad=True) for a in (hx, hz, w, cb, Wr, br, Wi, bi, lam)]
    y = om.gated_core(*args)
    y_c, _, _ = oracle.gated_forward(hx, hz, w, cb, Wr, br, Wi, bi, lam)
    np.testing.assert_allclose(y.detach().numpy(), y_c, rtol=1e-12, atol=1e-13)
    (y * torch.tensor(dy)).sum().backward()
    want = oracle.gated_backward(hx, hz, w, cb, Wr, br, Wi, bi, lam, dy)
    for a, k in zip(args, ("dhx", "dhz", "dconv_w", "dconv_b", "dWr", "dbr", "dWi", "dbi",
                           "dlambda")):
        np.testing.assert_allclose(a.grad.numpy(), want[k], rtol=1e-10, atol=1e-12, err_msg=k)


def test_layernorm_and_pffn_closed_forms():
    rng = np.random.default_rng(12)
    x = rng.standard_normal((3, 5, 8))
    y = om._ln(torch.tensor(x), torch.ones(8, dtype=torch.float64),
               torch.zeros(8, dtype=torch.float64), 0.0).numpy()
    np.testing.assert_allclose(y.mean(-1), 0.0, atol=1e-14)
    np.testing.assert_allclose((y ** 2).mean(-1), 1.0, rtol=1e-13)
    g, b = rng.standard_normal(8), rng.standard_normal(8)
    mu, var = x.mean(-1, keepdims=True), x.var(-1, keepdims=True)
    want = (x - mu) / np.sqrt(var + 1e-5) * g + b
    got = om._ln(torch.tensor(x), torch.tensor(g), torch.tensor(b), 1e-5).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-14)
    v = np.array([-3.0, -0.5, 0.0, 2.0])
    np.testing.assert_allclose(om._silu(torch.tensor(v)).numpy(), v * expit(v), rtol=1e-15)
    # softplus at points with known values: ln 2 at 0, ~v for large v, ~e^v for very negative v
    sp = om._softplus(torch.tensor([0.0, 40.0, -40.0], dtype=torch.float64)).numpy()
    np.testing.assert_allclose(sp, [np.log(2.0), 40.0, np.exp(-40.0)], rtol=1e-15)


def test_cross_entropy_closed_forms():
    """Equal item embeddings make every logit equal: loss = ln V exactly."""
    dims = TINY
    named, ids, targets = _setup()
    named["emb"] = np.tile(np.random.default_rng(13).standard_normal(dims.D), (dims.V, 1))
    assert abs(_loss(dims, named, ids, targets) - np.log(dims.V)) < 1e-12


def test_sublayers_zeroed_reduce_to_layernorms():
    """With Wo = 0, bo = 0 and W2 = 0, b2 = 0 every layer only re-normalises, so
    the last hidden state is a chain of LayerNorms of the embedding, written
    out here in numpy, and the loss is its cross entropy."""
    dims = TINY
    named, ids, targets = _setup(seed=7)
    for l in range(dims.layers):
        for k in ("Wo", "bo", "W2", "b2"):
            named[f"l{l}.{k}"] = np.zeros_like(named[f"l{l}.{k}"])

    def ln(x, g, b):
        mu, var = x.mean(-1, keepdims=True), x.var(-1, keepdims=True)
        return (x - mu) / np.sqrt(var + dims.eps) * g + b
    H = ln(named["emb"].astype(np.float64)[ids], named["emb_ln_g"], named["emb_ln_b"])
    for l in range(dims.layers):
        H = ln(H, named[f"l{l}.ln1_g"], named[f"l{l}.ln1_b"])
        H = ln(H, named[f"l{l}.ln2_g"], named[f"l{l}.ln2_b"])
    logits = H[:, -1] @ named["emb"].astype(np.float64).T
    want = np.mean(logsumexp(logits, axis=1) - logits[np.arange(dims.B), targets])
    assert abs(_loss(dims, named, ids, targets) - want) < 1e-12


def test_pffn_sublayer_written_out():
    """One layer with the gated recurrent layer's output zeroed: H2 = LN(H1 + PFFN(H1)),
    PFFN(H) = SiLU(H W1^T + b1) W2^T + b2 in numpy."""
    dims = dg.ModelDims(B=2, T=4, D=4, E=2, V=5, layers=1, K=2, eps=1e-5)
    named, ids, targets = _setup(dims, seed=8)
    named["l0.Wo"] = np.zeros_like(named["l0.Wo"])
    named["l0.bo"] = np.zeros_like(named["l0.bo"])
    f = lambda k: named[k].astype(np.float64)

    def ln(x, g, b):
        mu, var = x.mean(-1, keepdims=True), x.var(-1, keepdims=True)
        return (x - mu) / np.sqrt(var + dims.eps) * g + b
    H = ln(f("emb")[ids], f("emb_ln_g"), f("emb_ln_b"))
    H1 = ln(H, f("l0.ln1_g"), f("l0.ln1_b"))
    a = H1 @ f("l0.W1").T + f("l0.b1")
    H2 = ln(H1 + (a * expit(a)) @ f("l0.W2").T + f("l0.b2"), f("l0.ln2_g"), f("l0.ln2_b"))
    logits = H2[:, -1] @ f("emb").T
    want = np.mean(logsumexp(logits, axis=1) - logits[np.arange(dims.B), targets])
    assert abs(_loss(dims, named, ids, targets) - want) < 1e-12


@pytest.mark.parametrize("seed", [21, 22])
def test_model_gradient_central_differences(seed):
    """Gradient of the loss for a sample of every tensor against central differences."""
    dims = TINY
    named, ids, targets = _setup(seed=seed)
    flat = _flat(dims, named)
    loss, grad = om.train_step(flat, ids, targets, dims.D, dims.E, dims.V, dims.layers, dims.K,
                               dims.eps)
    assert abs(loss - _loss(dims, named, ids, targets)) < 1e-12
    lay, _ = om.layout(dims.D, dims.E, dims.V, dims.layers, dims.K)
    rng = np.random.default_rng(seed)
    eps = 1e-6
    for n, s, o in lay:
        size = int(np.prod(s))
        for k in rng.choice(size, size=min(3, size), replace=False):
            f2 = flat.copy()
            f2[o + k] += eps
            lp, _ = om.train_step(f2, ids, targets, dims.D, dims.E, dims.V, dims.layers,
                                  dims.K, dims.eps)
            f2[o + k] -= 2 * eps
            lm, _ = om.train_step(f2, ids, targets, dims.D, dims.E, dims.V, dims.layers,
                                  dims.K, dims.eps)
            fd = (lp - lm) / (2 * eps)
            assert abs(fd - grad[o + k]) <= 1e-6 * max(1.0, abs(fd)), (n, k, fd, grad[o + k])


def test_adam_first_step_closed_form():
    """Step 1: m_hat = g and v_hat = g^2, so the update is lr g / (|g| + eps)."""
    g = np.array([0.5, -2.0, 1e-3, 0.0])
    p = np.array([1.0, 1.0, 1.0, 1.0])
    m1, m2 = np.zeros(4), np.zeros(4)
    om.adam(p, g, m1, m2, 1, lr=0.01, eps=1e-8)
    np.testing.assert_allclose(p, 1.0 - 0.01 * g / (np.abs(g) + 1e-8), rtol=1e-14)


# ------------------------------------------------------------------ dropout and padding
def _numpy_u32(site, n, seed, offset):
    """32-bit words 0 .. n-1 of a dropout site from numpy's Philox4x64-10 bit
    generator: its first four outputs are the block at counter + 1, so the
    block at counter (g, site, 0, 0) comes from a generator started one below."""
    out = []
    for g in range(-(-n // 8)):
        ctr = (g + (site << 64) - 1) % 2 ** 256
        raw = np.random.Philox(counter=ctr, key=seed + (offset << 64)).random_raw(4)
        for w in raw:
            out += [int(w) & 0xFFFFFFFF, int(w) >> 32]
    return np.array(out[:n], dtype=np.uint64)


@pytest.mark.parametrize("ctr,key", [(0, 0), (1, 7), (2 ** 64 - 1, 2 ** 64 + 3),
                                     (12345 + (7 << 64) + (9 << 192), 2 ** 127 + 99)])
def test_philox_matches_numpy_bit_generator(ctr, key):
    """The oracle's Philox4x64-10 against numpy's implementation of the same
    generator (numpy.random.Philox), for counters that carry across words."""
    mask = 2 ** 64 - 1
    want = np.random.Philox(counter=(ctr - 1) % 2 ** 256, key=key).random_raw(4)
    got = om.philox4x64_10(*[(ctr >> (64 * i)) & mask for i in range(4)], key & mask,
                           key >> 64)
    assert [int(np.asarray(v)) for v in got] == [int(v) for v in want]


@pytest.mark.parametrize("site,n,seed,offset", [(0, 61, 1, 0), (3, 128, 2 ** 40 + 5, 17),
                                                 (6, 9, 0, 2 ** 63)])
def test_dropout_keep_from_numpy_words(site, n, seed, offset):
    """Element e of site s keeps iff its 32-bit word (numpy's generator) is at
    least floor(p 2^32); ragged n (not a multiple of 8) included."""
    u = _numpy_u32(site, n, seed, offset)
    for p in (0.0, 0.2, 0.5, 0.9):
        thr = int(np.floor(float(np.float32(p)) * 2.0 ** 32))
        np.testing.assert_array_equal(om.dropout_keep(site, n, p, seed, offset), u >= thr)


def test_dropout_threshold_and_rate():
    """floor(p 2^32) of the float32 p (0.2 is 13421773 * 2^-26 as a float32);
    the dropped fraction within 5 binomial deviations of p; sites and keys
    draw different masks."""
    assert om.drop_threshold(0.2) == 13421773 * 64
    assert om.drop_threshold(0.0) == 0 and om.drop_threshold(0.5) == 2 ** 31
    n = 400_000
    for p in (0.2, 0.5):
        drop = 1.0 - om.dropout_keep(1, n, p, 42, 3).mean()
        assert abs(drop - p) < 5 * np.sqrt(p * (1 - p) / n), (p, drop)
    a, b = om.dropout_keep(1, 4096, 0.5, 42, 3), om.dropout_keep(2, 4096, 0.5, 42, 3)
    c = om.dropout_keep(1, 4096, 0.5, 42, 4)
    assert 0.4 < (a == b).mean() < 0.6 and 0.4 < (a == c).mean() < 0.6


PAD = dg.ModelDims(B=3, T=6, D=4, E=2, V=9, layers=2, K=3, eps=1e-5)


def test_dropout_and_padding_forward_written_out():
    """Two layers with dropout p = 0.3 on the embedding and both sub-layer
    outputs and left-padded rows: the forward written out in numpy, with the
    gated recurrent core from the C oracle and the masks from numpy's
    generator, against the oracle's loss."""
    dims, p, seed, offset = PAD, 0.3, 11, 5
    named = dg.model_params(dims, 31)
    ids, targets = dg.model_batch(dims, 32, min_len=2, pad_id=0)
    assert (ids == 0).any() and (ids[:, -1] != 0).all()
    f = lambda k: named[k].astype(np.float64)
    scale = 1.0 / (1.0 - float(np.float32(p)))
    thr = int(np.floor(float(np.float32(p)) * 2.0 ** 32))

    def drop(x, site):
        keep = (_numpy_u32(site, x.size, seed, offset) >= thr).reshape(x.shape)
        return np.where(keep, x * scale, 0.0)

    def ln(x, g, b):
        mu, var = x.mean(-1, keepdims=True), x.var(-1, keepdims=True)
        return (x - mu) / np.sqrt(var + dims.eps) * g + b

    silu = lambda v: v * expit(v)
    X0 = f("emb")[ids] * (ids != 0)[..., None]
    H = ln(drop(X0, 0), f("emb_ln_g"), f("emb_ln_b"))
    for l in range(dims.layers):
        g = lambda k: f(f"l{l}.{k}")
        hx, hz = H @ g("Wx").T + g("bx"), H @ g("Wz").T + g("bz")
        y, _, _ = oracle.gated_forward(hx, hz, g("conv_w"), g("conv_b"), g("Wr"), g("br"),
                                       g("Wi"), g("bi"), g("lambda"))
        H1 = ln(H + drop(y @ g("Wo").T + g("bo"), 1 + 2 * l), g("ln1_g"), g("ln1_b"))
        H = ln(H1 + drop(silu(H1 @ g("W1").T + g("b1")) @ g("W2").T + g("b2"), 2 + 2 * l),
               g("ln2_g"), g("ln2_b"))
    logits = H[:, -1] @ f("emb").T
    want = np.mean(logsumexp(logits, axis=1) - logits[np.arange(dims.B), targets])
    pt = {k: torch.tensor(np.asarray(v, dtype=np.float64)) for k, v in named.items()}
    got = float(om.loss_fn(pt, torch.as_tensor(ids.astype(np.int64)),
                           torch.as_tensor(targets.astype(np.int64)), dims.D, dims.E, dims.V,
                           dims.layers, dims.K, dims.eps, dropout=p, seed=seed, offset=offset,
                           pad_id=0))
    assert abs(got - want) < 1e-12 * max(1.0, abs(want)), (got, want)


def test_padding_and_zero_dropout_special_cases():
    """p = 0 is no dropout whatever the key; a padding id that no position
    holds changes nothing; padded positions never read their row of E, so the
    hidden states do not move when E[pad] does, and dE[pad] is the prediction
    layer's part alone: sum_b (softmax(h_b E^T)[pad] - [target_b = pad]) h_b / B."""
    dims = PAD
    named = dg.model_params(dims, 33)
    flat = _flat(dims, named)
    ids, targets = dg.model_batch(dims, 34)
    args = (dims.D, dims.E, dims.V, dims.layers, dims.K, dims.eps)
    l0, g0 = om.train_step(flat, ids, targets, *args)
    l1, g1 = om.train_step(flat, ids, targets, *args, dropout=0.0, seed=9, offset=9)
    assert l0 == l1 and np.array_equal(g0, g1)
    free = np.setdiff1d(np.arange(dims.V), ids.ravel())
    assert free.size
    l2, g2 = om.train_step(flat, ids, targets, *args, pad_id=int(free[0]))
    assert l0 == l2 and np.array_equal(g0, g2)

    ids_p, targets_p = dg.model_batch(dims, 35, min_len=1, pad_id=0)
    assert (ids_p == 0).sum() > 0
    kw = dict(dropout=0.25, seed=3, offset=0, pad_id=0)
    tens = lambda nm: {k: torch.tensor(np.asarray(v, dtype=np.float64)) for k, v in nm.items()}
    ids_t = torch.as_tensor(ids_p.astype(np.int64))
    H = om.hidden(tens(named), ids_t, *args, **kw).numpy()
    moved = dict(named)
    moved["emb"] = named["emb"].copy()
    moved["emb"][0] = np.random.default_rng(36).standard_normal(dims.D) * 10
    assert np.array_equal(H, om.hidden(tens(moved), ids_t, *args, **kw).numpy())
    E = named["emb"].astype(np.float64)
    hT = H[:, -1]
    logits = hT @ E.T
    sm = np.exp(logits - logsumexp(logits, axis=1, keepdims=True))
    want = ((sm[:, 0] - (targets_p == 0)) @ hT) / dims.B
    _, gp = om.train_step(flat, ids_p, targets_p, *args, **kw)
    o_emb = om.layout(*args[:5])[0][0][2]
    np.testing.assert_allclose(gp[o_emb:o_emb + dims.D], want, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("seed", [23, 24])
def test_model_gradient_central_differences_dropout_padding(seed):
    """As the central-difference test above, with dropout 0.4 (fixed masks:
    the key is part of the input) and left-padded rows."""
    dims = PAD
    named = dg.model_params(dims, seed)
    ids, targets = dg.model_batch(dims, seed + 1, min_len=2, pad_id=0)
    flat = _flat(dims, named)
    kw = dict(dropout=0.4, seed=seed, offset=1, pad_id=0)
    args = (dims.D, dims.E, dims.V, dims.layers, dims.K, dims.eps)
    loss, grad = om.train_step(flat, ids, targets, *args, **kw)
    lay, _ = om.layout(*args[:5])
    rng = np.random.default_rng(seed)
    eps = 1e-6
    for n, s, o in lay:
        size = int(np.prod(s))
        for k in rng.choice(size, size=min(3, size), replace=False):
            f2 = flat.copy()
            f2[o + k] += eps
            lp, _ = om.train_step(f2, ids, targets, *args, **kw)
            f2[o + k] -= 2 * eps
            lm, _ = om.train_step(f2, ids, targets, *args, **kw)
            fd = (lp - lm) / (2 * eps)
            assert abs(fd - grad[o + k]) <= 1e-6 * max(1.0, abs(fd)), (n, k, fd, grad[o + k])
