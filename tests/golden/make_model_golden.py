"""Writes tests/golden/model_ml1m_oracle.npz: the fp64 oracle's loss and
gradients of one training step of the full model at the MovieLens-1M training
shape (section 4.1 implementation details: batch 2048, maximum length 200,
D = 64, expansion factor 2, two layers, 3,416 items).

The oracle (oracle/model.py, plain PyTorch CPU float64) takes minutes and tens
of GB at this shape, so its result is stored; the GPU test regenerates the
same seeded inputs with paper_2406_12580_amd.datagen and compares.  Nothing
here calls the HIP library.  Run from the repository root:
    python tests/golden/make_model_golden.py
"""
import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import model as om  # noqa: E402
from paper_2406_12580_amd import datagen as dg  # noqa: E402

NAME, PARAM_SEED, BATCH_SEED = "ml1m", 700, 800
OUT = os.path.join(HERE, "model_ml1m_oracle.npz")


def inputs():
    """The seeded parameters (flat, oracle layout, float64), ids and targets."""
    d = dg.MODEL_CONFIGS[NAME]
    named = dg.model_params(d, PARAM_SEED)
    ids, targets = dg.model_batch(d, BATCH_SEED)
    lay, total = om.layout(d.D, d.E, d.V, d.layers, d.K)
    flat = np.zeros(total)
    for n, s, o in lay:
        flat[o:o + int(np.prod(s))] = named[n].astype(np.float64).ravel()
    return d, named, ids, targets, flat


def fingerprint(flat, ids, targets):
    """sha256 of the inputs, so the test can tell that datagen still draws them."""
    h = hashlib.sha256()
    for a in (flat.astype(np.float64), ids.astype(np.int32), targets.astype(np.int32)):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def main():
    d, _, ids, targets, flat = inputs()
    t0 = time.time()
    loss, grads = om.train_step(flat, ids, targets, d.D, d.E, d.V, d.layers, d.K, d.eps)
    print(f"oracle step at {d}: loss {loss:.6f}, {time.time() - t0:.0f} s")
    # The gradients are stored rounded to float32: a relative change below
    # 6e-8, far inside the 1e-4 bar they are checked against.
    np.savez_compressed(OUT, loss=np.float64(loss), grads=grads.astype(np.float32),
                        fingerprint=np.array(fingerprint(flat, ids, targets)))


if __name__ == "__main__":
    main()
