"""Writes tests/golden/oracle_small.json from the fp64 oracle alone.

This is a regression fixture for the oracle (a drift detector), not a pin:
the pins are the closed forms, brute force, two-tree scan and finite
differences in tests/test_oracle_pins.py.  Run from the repository root:
    python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2406_12580_amd import datagen as dg  # noqa: E402

SHAPE, SEED = (2, 6, 3), 31


def main():
    inp = dg.scan_inputs(*SHAPE, seed=SEED, h0=True, grad=True, dhT=True)
    h, hT = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
    bw = oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh, inp.h0, inp.dhT)
    out = {"shape": list(SHAPE), "seed": SEED, "h": h.ravel().tolist(), "hT": hT.ravel().tolist()}
    for k in ("dx", "dzr", "dzi", "dlambda", "dh0"):
        out[k] = bw[k].ravel().tolist()
    with open(os.path.join(HERE, "oracle_small.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
