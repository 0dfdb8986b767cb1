"""recblr_bdlru_scan_backward_noalloc: the scan backward on the library's
static device scratch (no workspace argument, nothing allocated) against
recblr_bdlru_scan_backward with a caller's workspace, through the C ABI.

Calls run back to back on the shared static array, each followed by a
smaller problem, so that whatever a call leaves in the array (look-back
state words, ticket, dLambda partials) would show up in the next one: every
output must equal the workspace entry point's bit for bit (both run the same
kernels), and match the fp64 oracle within the fp32 / bf16 bar.
"""
import numpy as np
import pytest

import oracle
from helpers import assert_close, dev, dev32, host
from paper_2406_12580_amd import datagen as dg

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rb():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2406_12580_amd import recblr
    return recblr


def _both(rb, inp, with_state):
    """(noalloc outputs, workspace outputs) of one problem, as host arrays."""
    import torch
    io = inp.io
    B, L, D = inp.x.shape
    X, ZR, ZI, DH = (dev(a, io) for a in (inp.x, inp.zr, inp.zi, inp.dh))
    lam = dev32(inp.lam)
    h0 = dev32(inp.h0) if with_state else None
    dhT = dev32(inp.dhT) if with_state else None
    h, _ = rb.bdlru_scan_forward(X, ZR, ZI, lam, h0)
    code = rb.io_code(X.dtype)
    p = lambda t: None if t is None else t.data_ptr()
    s = torch.cuda.current_stream().cuda_stream
    res = []
    for noalloc in (True, False):
        o = {k: torch.full_like(X, float("nan")) for k in ("dx", "dzr", "dzi")}
        o["dlambda"] = torch.full((D,), float("nan"), device=X.device)
        o["dh0"] = torch.full((B, D), float("nan"), device=X.device)
        args = (p(X), p(ZR), p(ZI), p(lam), p(h0), p(h), p(DH), p(dhT), p(o["dx"]), p(o["dzr"]),
                p(o["dzi"]), p(o["dlambda"]), p(o["dh0"]), B, L, D, code)
        if noalloc:
            st = rb.recblr_bdlru_scan_backward_noalloc(*args, s)
        else:
            nws = rb.recblr_workspace_size(rb.OP_SCAN_BACKWARD, B, L, D, code)
            ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=X.device)
            st = rb.recblr_bdlru_scan_backward(*args, p(ws), nws, s)
        assert st == 0, rb.recblr_status_string(st)
        torch.cuda.synchronize()
        res.append({k: host(v) for k, v in o.items()})
    return res


# Pairs of calls in a row: a larger problem, then a smaller one.  Look-back
# shapes (few channel groups, long sequences) use the state words and the
# ticket; the chain shape only the dLambda partials.
PAIRS = [
    (((2, 3000, 256), "bf16"), ((1, 700, 64), "bf16")),
    (((1, 5000, 64), "f32"), ((3, 300, 40), "f32")),
    (((64, 300, 512), "f32"), ((2, 1, 64), "f32")),
]


@pytest.mark.parametrize("pair", range(len(PAIRS)))
def test_noalloc_matches_workspace_entry_point(rb, pair):
    for k, (shape, io) in enumerate(PAIRS[pair]):
        B, L, D = shape
        inp = dg.scan_inputs(B, L, D, 9800 + 10 * pair + k, io=io, h0=True, grad=True, dhT=True)
        got, ref = _both(rb, inp, True)
        print(f"noalloc {shape} {io}: GPU done", flush=True)
        for name in got:
            assert np.array_equal(got[name].view(np.uint32), ref[name].view(np.uint32)), name
        want = oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh, inp.h0, inp.dhT)
        for name in ("dx", "dzr", "dzi", "dlambda"):
            assert_close(got[name], want[name], io, name)
        assert_close(got["dh0"], want["dh0"], "f32", "dh0")


def test_noalloc_full_size_then_smaller(rb):
    """The long-history workload at full size (6 MiB of the static scratch),
    then a small problem on the same array."""
    cfg = dg.CONFIGS["c4"]
    inp = dg.config_inputs(cfg, grad=True)
    got, ref = _both(rb, inp, False)
    print("noalloc c4: GPU done", flush=True)
    for name in got:
        assert np.array_equal(got[name].view(np.uint32), ref[name].view(np.uint32)), name
    small = dg.scan_inputs(4, 50, 64, 9850, h0=True, grad=True, dhT=True)
    got, ref = _both(rb, small, True)
    for name in got:
        assert np.array_equal(got[name].view(np.uint32), ref[name].view(np.uint32)), name
    want = oracle.scan_backward(small.x, small.zr, small.zi, small.lam, small.dh, small.h0,
                                small.dhT)
    for name in ("dx", "dzr", "dzi", "dlambda", "dh0"):
        assert_close(got[name], want[name], "f32", name)
