"""Writes the fp64 oracle's loss and gradients of one training step of the
full model at the MovieLens-1M training shape (section 4.1 implementation
details: batch 2048, maximum length 200, D = 64, expansion factor 2, two
layers, 3,416 items), for two batches:
  tests/golden/model_ml1m_oracle.npz          full-length rows, no dropout;
  tests/golden/model_ml1m_dropout_oracle.npz  the dataset's length mix
      (lengths U{131..200}, mean 165.5 as in table tab:dataset, left-padded
      with id 0) and dropout 0.2 (the rate the dropout study finds best for
      MovieLens-1M), Philox key (2406, 1).

The oracle (oracle/model.py, plain PyTorch CPU float64) takes minutes and tens
of GB at this shape, so its result is stored; the GPU test regenerates the
same seeded inputs with paper_2406_12580_amd.datagen and compares.  Nothing
here calls the HIP library.  Run from the repository root:
    python tests/golden/make_model_golden.py [ml1m | ml1m-dropout]
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
# variant: (output file, model_batch keywords, train-step options)
VARIANTS = {
    "ml1m": ("model_ml1m_oracle.npz", {}, {}),
    "ml1m-dropout": ("model_ml1m_dropout_oracle.npz",
                     {"min_len": dg.ml1m_min_len(), "pad_id": 0},
                     {"dropout": 0.2, "seed": 2406, "offset": 1, "pad_id": 0}),
}


def path(variant="ml1m"):
    return os.path.join(HERE, VARIANTS[variant][0])


def options(variant="ml1m"):
    """Dropout probability, Philox key and padding id of the variant's step."""
    return dict(VARIANTS[variant][2])


def inputs(variant="ml1m"):
    """The seeded parameters (flat, oracle layout, float64), ids and targets."""
    d = dg.MODEL_CONFIGS[NAME]
    named = dg.model_params(d, PARAM_SEED)
    ids, targets = dg.model_batch(d, BATCH_SEED, **VARIANTS[variant][1])
    lay, total = om.layout(d.D, d.E, d.V, d.layers, d.K)
    flat = np.zeros(total)
    for n, s, o in lay:
        flat[o:o + int(np.prod(s))] = named[n].astype(np.float64).ravel()
    return d, named, ids, targets, flat


def fingerprint(flat, ids, targets, opts=None):
    """sha256 of the inputs, so the test can tell that datagen still draws them."""
    h = hashlib.sha256()
    for a in (flat.astype(np.float64), ids.astype(np.int32), targets.astype(np.int32)):
        h.update(np.ascontiguousarray(a).tobytes())
    if opts:
        h.update(repr(sorted(opts.items())).encode())
    return h.hexdigest()


def main(variant="ml1m"):
    d, _, ids, targets, flat = inputs(variant)
    opts = options(variant)
    t0 = time.time()
    loss, grads = om.train_step(flat, ids, targets, d.D, d.E, d.V, d.layers, d.K, d.eps, **opts)
    print(f"oracle step at {d} {opts}: loss {loss:.6f}, {time.time() - t0:.0f} s")
    # The gradients are stored rounded to float32: a relative change below
    # 6e-8, far inside the 1e-4 bar they are checked against.
    np.savez_compressed(path(variant), loss=np.float64(loss), grads=grads.astype(np.float32),
                        fingerprint=np.array(fingerprint(flat, ids, targets, opts)))


if __name__ == "__main__":
    main(*sys.argv[1:2])
