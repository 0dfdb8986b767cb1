"""GPU parity of the full RecBLR model training step (recblr_model_train_step,
recblr_adam_update) against the fp64 oracle of oracle/model.py.

Every gradient tensor is compared with the floored relative error of the
other parity tests at the fp32 bar (1e-4).
"""
import os
import sys

import numpy as np
import pytest

from helpers import assert_close, report
from oracle import model as om
from paper_2406_12580_amd import datagen as dg

pytestmark = pytest.mark.gpu

CASES = [dg.MODEL_CONFIGS["ml1m-small"],
         dg.ModelDims(B=2, T=5, D=128, E=1, V=37, layers=1, K=2, eps=1e-5),
         dg.ModelDims(B=3, T=70, D=64, E=3, V=300, layers=3, K=4, eps=1e-6),
         # 8,320 rows: weight gradients in chunks of 4,096 rows plus a remainder;
         # popular items span several 256-position pieces of the embedding gradient
         dg.ModelDims(B=64, T=130, D=64, E=2, V=500, layers=1, K=4)]


@pytest.fixture(scope="module")
def rb():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2406_12580_amd import recblr
    return recblr


def _device_params(rb, dims, named):
    import torch
    rd = rb.model_dims(dims.B, dims.T, dims.D, dims.E, dims.V, dims.layers, dims.K, dims.eps)
    offs = rb.model_param_offsets(rd)
    lay, total = om.layout(dims.D, dims.E, dims.V, dims.layers, dims.K)
    flat = np.zeros(rb.recblr_model_param_count(rd), dtype=np.float32)
    for (name, shape, _), o in zip(lay, offs):
        flat[o:o + int(np.prod(shape))] = named[name].ravel()
    return rd, torch.from_numpy(flat).cuda(), flat


# Dropout and padding: (dims, shortest row length or None for full rows,
# drop probability, padding id, Philox seed, Philox offset).
DROP_CASES = [
    (dg.MODEL_CONFIGS["ml1m-small"], 5, 0.2, 0, 7, 3),
    (dg.ModelDims(B=2, T=5, D=128, E=1, V=37, layers=1, K=2, eps=1e-5), None, 0.1, -1, 1, 0),
    (dg.ModelDims(B=3, T=70, D=64, E=3, V=300, layers=3, K=4, eps=1e-6), 1, 0.5, 0,
     2 ** 40 + 1, 2 ** 63),
    (dg.ModelDims(B=2, T=9, D=256, E=1, V=40, layers=1, K=3, eps=1e-5), 2, 0.3, 0, 5, 6),
    (dg.ModelDims(B=5, T=33, D=64, E=2, V=90, layers=2, K=4, eps=1e-5), 3, 0.0, 0, 0, 0),
    (dg.ModelDims(B=64, T=130, D=64, E=2, V=500, layers=1, K=4), 20, 0.2, 0, 11, 12),
]


def _oracle_flat(dims, named):
    lay, total = om.layout(dims.D, dims.E, dims.V, dims.layers, dims.K)
    flat = np.zeros(total)
    for n, s, o in lay:
        flat[o:o + int(np.prod(s))] = named[n].astype(np.float64).ravel()
    return flat, lay


@pytest.mark.parametrize("case", range(len(CASES)))
def test_model_train_step(rb, case):
    import torch
    dims = CASES[case]
    named = dg.model_params(dims, 700 + case)
    ids, targets = dg.model_batch(dims, 800 + case)
    rd, P, _ = _device_params(rb, dims, named)
    step = rb.ModelStep(rd)
    I, Tg = torch.from_numpy(ids).cuda(), torch.from_numpy(targets).cuda()
    loss, grads = step.train_step(P, I, Tg)
    loss2, grads2 = step.train_step(P, I, Tg)
    torch.cuda.synchronize()
    print(f"model step {dims}: GPU done", flush=True)
    g = grads.cpu().numpy()
    assert np.array_equal(g.view(np.uint32), grads2.cpu().numpy().view(np.uint32)), \
        "gradients must repeat bitwise"
    assert loss.item() == loss2.item()
    flat, lay = _oracle_flat(dims, named)
    want_loss, want = om.train_step(flat, ids, targets, dims.D, dims.E, dims.V, dims.layers,
                                    dims.K, dims.eps)
    assert abs(loss.item() - want_loss) <= 1e-4 * abs(want_loss), (loss.item(), want_loss)
    offs = rb.model_param_offsets(rd)
    for (name, shape, o_ref), o in zip(lay, offs):
        n = int(np.prod(shape))
        assert_close(g[o:o + n], want[o_ref:o_ref + n], "f32", name)
    # padding between tensors stays zero
    mask = np.ones(g.size, dtype=bool)
    for (name, shape, _), o in zip(lay, offs):
        mask[o:o + int(np.prod(shape))] = False
    assert not g[mask].any()
    step.close()


def _check_against_oracle(rb, rd, dims, g, loss, want_loss, want, tag=""):
    assert abs(loss - want_loss) <= 1e-4 * abs(want_loss), (loss, want_loss)
    lay, _ = om.layout(dims.D, dims.E, dims.V, dims.layers, dims.K)
    offs = rb.model_param_offsets(rd)
    for (name, shape, o_ref), o in zip(lay, offs):
        n = int(np.prod(shape))
        if tag:
            report(f"{tag} {name}", g[o:o + n], want[o_ref:o_ref + n])
        assert_close(g[o:o + n], want[o_ref:o_ref + n], "f32", name)


@pytest.mark.parametrize("case", range(len(DROP_CASES)))
def test_model_train_step_dropout_padding(rb, case):
    """Dropout (masks from the counter-based generator, drawn on the GPU) and
    left-padded rows: every gradient against the oracle's, bitwise repeats for
    one key, new masks for a new offset."""
    import torch
    dims, min_len, p, pad, seed, offset = DROP_CASES[case]
    named = dg.model_params(dims, 900 + case)
    if min_len is None:
        ids, targets = dg.model_batch(dims, 950 + case)
    else:
        ids, targets = dg.model_batch(dims, 950 + case, min_len=min_len, pad_id=pad)
        assert (ids == pad).any()
    rd, P, _ = _device_params(rb, dims, named)
    step = rb.ModelStep(rd)
    I, Tg = torch.from_numpy(ids).cuda(), torch.from_numpy(targets).cuda()
    kw = dict(dropout=p, seed=seed, offset=offset, pad_id=pad)
    loss, grads = step.train_step(P, I, Tg, **kw)
    loss2, grads2 = step.train_step(P, I, Tg, **kw)
    loss3, grads3 = step.train_step(P, I, Tg, **dict(kw, offset=offset + 1))
    torch.cuda.synchronize()
    print(f"model step {dims} {kw}: GPU done", flush=True)
    g = grads.cpu().numpy()
    assert np.array_equal(g.view(np.uint32), grads2.cpu().numpy().view(np.uint32))
    assert loss.item() == loss2.item()
    if p > 0:
        assert not np.array_equal(g, grads3.cpu().numpy()), "a new offset must draw new masks"
    flat, _ = _oracle_flat(dims, named)
    want_loss, want = om.train_step(flat, ids, targets, dims.D, dims.E, dims.V, dims.layers,
                                    dims.K, dims.eps, **kw)
    _check_against_oracle(rb, rd, dims, g, loss.item(), want_loss, want)
    step.close()


def test_adam_update(rb):
    import torch
    rng = np.random.default_rng(5)
    n = 1000
    p, g = rng.standard_normal(n).astype(np.float32), rng.standard_normal(n).astype(np.float32)
    m1, m2 = (rng.standard_normal(n) * 0.1).astype(np.float32), \
        np.abs(rng.standard_normal(n) * 0.01).astype(np.float32)
    P, G, M1, M2 = (torch.from_numpy(a.copy()).cuda() for a in (p, g, m1, m2))
    rb.adam_update(P, G, M1, M2, 7, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)
    torch.cuda.synchronize()
    pr, m1r, m2r = (a.astype(np.float64) for a in (p, m1, m2))
    # the hyper-parameters the library received: their float32 values, widened exactly
    f = lambda v: float(np.float32(v))
    om.adam(pr, g.astype(np.float64), m1r, m2r, 7, lr=f(1e-3), beta1=f(0.9), beta2=f(0.999),
            eps=f(1e-8))
    # fp32 against fp64: each result within a few ulp of its largest operand
    # (|p| below 4, |0.9 m1| and |0.1 g| below 0.4, m2 below 0.05).
    ulp = 2.0 ** -23
    np.testing.assert_allclose(P.cpu().numpy(), pr, rtol=8 * ulp, atol=4 * 4 * ulp)
    np.testing.assert_allclose(M1.cpu().numpy(), m1r, rtol=8 * ulp, atol=4 * 0.4 * ulp)
    np.testing.assert_allclose(M2.cpu().numpy(), m2r, rtol=8 * ulp, atol=4 * 0.05 * ulp)


def test_out_of_range_ids_give_nan_loss(rb):
    """An item id or target outside [0, V) is read as row 0 and makes the loss NaN."""
    import torch
    dims = dg.ModelDims(B=2, T=6, D=64, E=2, V=50, layers=1, K=4, eps=1e-5)
    named = dg.model_params(dims, 9)
    ids, targets = dg.model_batch(dims, 10)
    rd, P, _ = _device_params(rb, dims, named)
    step = rb.ModelStep(rd)
    bad_ids = ids.copy()
    bad_ids[1, 3] = dims.V
    loss, _ = step.train_step(P, torch.from_numpy(bad_ids).cuda(), torch.from_numpy(targets).cuda())
    bad_t = targets.copy()
    bad_t[0] = -1
    loss2, _ = step.train_step(P, torch.from_numpy(ids).cuda(), torch.from_numpy(bad_t).cuda())
    torch.cuda.synchronize()
    assert np.isnan(loss.item()) and np.isnan(loss2.item())
    step.close()


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "model_ml1m_oracle.npz")


@pytest.mark.parametrize("variant", ["ml1m", "ml1m-dropout"])
def test_model_train_step_ml1m(rb, variant):
    """The MovieLens-1M training shape the model bench times (batch 2048,
    length 200, D = 64, E = 2, two layers, 3,416 items), with full-length rows
    and no dropout, and with the dataset's length mix (left-padded) and
    dropout 0.2: every gradient tensor against the fp64 oracle's, stored by
    tests/golden/make_model_golden.py (the oracle takes minutes at this size)
    for the same seeded inputs."""
    import torch
    sys.path.insert(0, os.path.dirname(GOLDEN))
    import make_model_golden as mg
    dims, named, ids, targets, flat64 = mg.inputs(variant)
    opts = mg.options(variant)
    golden = np.load(mg.path(variant), allow_pickle=False)
    assert str(golden["fingerprint"]) == mg.fingerprint(flat64, ids, targets, opts), \
        "the seeded inputs changed since the oracle result was stored"
    rd, P, _ = _device_params(rb, dims, named)
    step = rb.ModelStep(rd)
    loss, grads = step.train_step(P, torch.from_numpy(ids).cuda(),
                                  torch.from_numpy(targets).cuda(), **opts)
    torch.cuda.synchronize()
    print(f"model step {dims} {opts}: GPU done", flush=True)
    _check_against_oracle(rb, rd, dims, grads.cpu().numpy(), loss.item(), float(golden["loss"]),
                          golden["grads"].astype(np.float64), tag=f"model {variant}")
    step.close()
