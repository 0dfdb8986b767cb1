"""GPU parity of every librecblr.so entry point against the fp64 oracle.

All inputs come from paper_2406_12580_amd.datagen (seeded); the GPU path is
called through the C ABI (ctypes binding) and compared element by element with
the oracle under the floored relative error of tests/helpers.py
(1e-4 for fp32 I/O, 1e-2 for bf16 I/O).  Shapes cover several macro-chunks of
the scan kernels with ragged tails, channel groups that span batch rows
(D < 64 and D not a multiple of 64), L = 1, D = 1 and the degenerate L = 0 and
B = 0 cases; the named workloads run at full size with every element compared.
"""
import numpy as np
import pytest

import oracle
from helpers import TOL, assert_close, dev, dev32, floored_rel_err, host, report
from paper_2406_12580_amd import datagen as dg

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rb():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2406_12580_amd import recblr
    return recblr


SHAPES = [(4, 50, 64), (3, 131, 48), (2, 1, 64), (1, 2, 1), (5, 257, 72), (2, 97, 3),
          (3, 513, 130), (1, 64, 128)]


def _run_fwd(rb, inp):
    return rb.bdlru_scan_forward(dev(inp.x, inp.io), dev(inp.zr, inp.io), dev(inp.zi, inp.io),
                                 dev32(inp.lam), dev32(inp.h0))


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_scan_forward(rb, shape, io):
    B, L, D = shape
    seed = 1000 + B * 7 + L * 13 + D
    for with_h0 in (False, True):
        inp = dg.scan_inputs(B, L, D, seed, io=io, h0=with_h0)
        h, hT = _run_fwd(rb, inp)
        oh, ohT = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
        print(f"scan_forward {shape} {io} h0={with_h0}", flush=True)
        assert_close(host(h), oh, io, "h")
        assert_close(host(hT), ohT, "f32", "hT")  # the fp32 state: fp32 bar for both I/O types


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_scan_backward(rb, shape, io):
    B, L, D = shape
    inp = dg.scan_inputs(B, L, D, 2000 + B + L + D, io=io, h0=True, grad=True, dhT=True)
    X, ZR, ZI = dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io)
    lam, h0 = dev32(inp.lam), dev32(inp.h0)
    h, _ = rb.bdlru_scan_forward(X, ZR, ZI, lam, h0)
    got = rb.bdlru_scan_backward(X, ZR, ZI, lam, h, dev(inp.dh, io), h0, dev32(inp.dhT))
    want = oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh, inp.h0, inp.dhT)
    print(f"scan_backward {shape} {io}", flush=True)
    for k in ("dx", "dzr", "dzi", "dlambda"):
        assert_close(host(got[k]), want[k], io, k)
    assert_close(host(got["dh0"]), want["dh0"], "f32", "dh0")  # fp32 adjoint state


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_scan_variants(rb, io):
    """SiLU-shaped x, nonzero h0, extreme decay bases and left-zero-padded rows."""
    cases = [dict(silu_x=True, h0=True), dict(a_range=(0.5, 0.9)),
             dict(a_range=(0.9999, 0.99999)), dict(pad_rows=True)]
    for k, kw in enumerate(cases):
        inp = dg.scan_inputs(6, 300, 64, 3000 + k, io=io, **kw)
        h, hT = _run_fwd(rb, inp)
        oh, ohT = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
        assert_close(host(h), oh, io, f"h {kw}")
        if kw.get("pad_rows"):
            lengths = inp.extra["lengths"]
            hh = host(h)
            for b in range(6):
                assert np.all(hh[b, : 300 - lengths[b]] == 0.0)  # exact zeros before the row starts


def test_alpha_to_zero_gives_gated_input(rb):
    inp = dg.scan_inputs(3, 70, 64, 3100, h0=True)
    inp.lam[:] = 1000.0
    inp.zr[:] = 40.0
    h, _ = _run_fwd(rb, inp)
    i = 1.0 / (1.0 + np.exp(-inp.zi.astype(np.float64)))
    assert_close(host(h), i * inp.x, "f32", "h")


def test_linear_scan_closed_forms(rb):
    import torch
    rng = np.random.Generator(np.random.PCG64(3200))
    B, L, D = 3, 333, 70
    u = rng.standard_normal((B, L, D), dtype=np.float32)
    h0 = rng.standard_normal((B, D), dtype=np.float32)
    h, hT = rb.linear_scan_forward(dev32(np.zeros_like(u)), dev32(u), dev32(h0))
    np.testing.assert_array_equal(host(h), u)                     # a = 0: h = u exactly
    h, hT = rb.linear_scan_forward(dev32(np.ones_like(u)), dev32(u), dev32(h0))
    want = h0[:, None, :].astype(np.float64) + np.cumsum(u.astype(np.float64), axis=1)
    assert_close(host(h), want, "f32", "prefix sum")
    a = np.broadcast_to(np.float32(0.9), (B, L, D)).copy()
    c = np.full((B, L, D), 0.5, np.float32)
    h, hT = rb.linear_scan_forward(dev32(a), dev32(c), dev32(h0))
    t = np.arange(1, L + 1)[None, :, None]
    aa = np.float64(np.float32(0.9))
    want = aa ** t * h0[:, None, :] + 0.5 * (1 - aa ** t) / (1 - aa)
    assert_close(host(h), want, "f32", "geometric")
    a = rng.uniform(0, 1.1, (B, L, D)).astype(np.float32)
    h, hT = rb.linear_scan_forward(dev32(a), dev32(u), dev32(h0))
    oh, ohT = oracle.linear_scan(a, u, h0)
    assert_close(host(h), oh, "f32", "raw")
    assert_close(host(hT), ohT, "f32", "raw hT")
    torch.cuda.synchronize()


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("B,D", [(65, 256), (7, 3), (3, 2056), (33, 64)])
def test_scan_step(rb, io, B, D):
    inp = dg.step_inputs(B, D, 3300 + B + D, io=io)
    got = rb.bdlru_scan_step(dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io), dev32(inp.lam),
                             dev32(inp.h0))
    want = oracle.scan_step(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
    assert_close(host(got), want, io, "h_next")
    # in place: h_next aliases h_prev
    hp = dev32(inp.h0)
    rb.bdlru_scan_step(dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io), dev32(inp.lam), hp,
                       out=hp)
    assert_close(host(hp), want, io, "h_next in place")


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_steps_equal_scan(rb, io):
    inp = dg.scan_inputs(5, 40, 96, 3400, io=io, h0=True)
    h, _ = _run_fwd(rb, inp)
    import torch
    state = dev32(inp.h0)
    X, ZR, ZI = dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io)
    lam = dev32(inp.lam)
    for t in range(40):
        state = rb.bdlru_scan_step(X[:, t].contiguous(), ZR[:, t].contiguous(),
                                   ZI[:, t].contiguous(), lam, state)
    torch.cuda.synchronize()
    oh, _ = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
    assert_close(host(state), oh[:, -1], io, "stepped state")


def test_split_and_continue(rb):
    inp = dg.scan_inputs(4, 700, 64, 3500, h0=True)
    m = 333
    X, ZR, ZI, lam = dev(inp.x), dev(inp.zr), dev(inp.zi), dev32(inp.lam)
    h, hT = rb.bdlru_scan_forward(X, ZR, ZI, lam, dev32(inp.h0))
    h1, hm = rb.bdlru_scan_forward(X[:, :m].contiguous(), ZR[:, :m].contiguous(),
                                   ZI[:, :m].contiguous(), lam, dev32(inp.h0))
    h2, hT2 = rb.bdlru_scan_forward(X[:, m:].contiguous(), ZR[:, m:].contiguous(),
                                    ZI[:, m:].contiguous(), lam, hm)
    oh, _ = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
    assert_close(np.concatenate([host(h1), host(h2)], axis=1), oh, "f32", "split")
    assert floored_rel_err(host(hT2), host(hT)) <= 1e-5


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_empty_and_degenerate(rb, io):
    import torch
    inp = dg.scan_inputs(3, 0, 8, 3600, io=io, h0=True, grad=True, dhT=True)
    h, hT = _run_fwd(rb, inp)
    assert h.shape == (3, 0, 8)
    np.testing.assert_array_equal(host(hT), inp.h0)                   # L = 0: hT = h0
    X, ZR, ZI = dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io)
    got = rb.bdlru_scan_backward(X, ZR, ZI, dev32(inp.lam), dev(inp.x, io), dev(inp.x, io),
                                 dev32(inp.h0), dev32(inp.dhT))
    np.testing.assert_array_equal(host(got["dh0"]), inp.dhT)
    np.testing.assert_array_equal(host(got["dlambda"]), 0.0)
    # B = 0: nothing to compute; dLambda is an empty sum
    inp0 = dg.scan_inputs(0, 5, 8, 3601, io=io, grad=True)
    h, hT = _run_fwd(rb, inp0)
    assert h.shape == (0, 5, 8)
    X0 = dev(inp0.x, io)
    got = rb.bdlru_scan_backward(X0, X0, X0, dev32(inp0.lam), X0, X0)
    np.testing.assert_array_equal(host(got["dlambda"]), 0.0)
    torch.cuda.synchronize()


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_deterministic(rb, io):
    inp = dg.scan_inputs(16, 300, 64, 3700, io=io, h0=True, grad=True, dhT=True)
    X, ZR, ZI, lam, h0 = dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io), dev32(inp.lam), \
        dev32(inp.h0)
    outs = []
    for _ in range(2):
        h, hT = rb.bdlru_scan_forward(X, ZR, ZI, lam, h0)
        g = rb.bdlru_scan_backward(X, ZR, ZI, lam, h, dev(inp.dh, io), h0, dev32(inp.dhT))
        outs.append([host(h), host(hT)] + [host(g[k]) for k in sorted(g)])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)


# ------------------------------------------------------------------ entry points with gate parameters

@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(2, 37, 64), (3, 70, 48), (1, 5, 130), (2, 130, 256)])
def test_full_forward_backward(rb, shape, io):
    B, L, D = shape
    f = dg.full_inputs(B, L, D, 4000 + B + L + D, io=io, bias=True, h0=True, grad=True, dhT=True)
    X, Wr, br, Wi, bi = (dev(a, io) for a in (f.x, f.Wr, f.br, f.Wi, f.bi))
    lam, h0 = dev32(f.lam), dev32(f.h0)
    h, hT = rb.bdlru_forward(X, Wr, br, Wi, bi, lam, h0)
    oh, ohT = oracle.forward(f.x, f.Wr, f.br, f.Wi, f.bi, f.lam, f.h0)
    print(f"full {shape} {io}", flush=True)
    assert_close(host(h), oh, io, "h")
    assert_close(host(hT), ohT, io, "hT")
    got = rb.bdlru_backward(X, Wr, br, Wi, bi, lam, h, dev(f.dh, io), h0, dev32(f.dhT))
    want = oracle.backward(f.x, f.Wr, f.br, f.Wi, f.bi, f.lam, f.dh, f.h0, f.dhT)
    for k in ("dx", "dWr", "dbr", "dWi", "dbi", "dlambda", "dh0"):
        assert_close(host(got[k]), want[k], io, k)


# With D % 64 == 0 the forward and the backward recompute the gate
# projections inside the look-back scan (tiles of 64 channels x 128 steps);
# these shapes span several tiles with a ragged last one.  D = 72 takes the
# path through the separate projection kernels.
FUSED_FWD = [(1, 1000, 64), (3, 700, 128), (2, 257, 192), (1, 129, 256), (2, 1000, 72),
             # D = 128 / 256 with W kept in registers: few channel groups take
             # tiles in ticket order with look-back (above), at least 256 groups
             # walk their tiles in a chain (below; ragged last tile, L = 1)
             (256, 100, 128), (512, 1, 128), (128, 77, 256),
             # many tiles per group: the workgroups' tickets run several tiles
             # ahead of the one they work on
             (2, 4100, 256), (5, 3000, 128)]


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("shape", FUSED_FWD)
def test_full_forward_fused(rb, shape, io):
    B, L, D = shape
    f = dg.full_inputs(B, L, D, 4300 + B + L + D, io=io, a_range=(0.99, 0.9999), bias=True,
                       h0=True)
    h, hT = rb.bdlru_forward(*(dev(a, io) for a in (f.x, f.Wr, f.br, f.Wi, f.bi)),
                             dev32(f.lam), dev32(f.h0))
    print(f"fused forward {shape} {io}: GPU done", flush=True)
    oh, ohT = oracle.forward(f.x, f.Wr, f.br, f.Wi, f.bi, f.lam, f.h0)
    assert_close(host(h), oh, io, "h")
    assert_close(host(hT), ohT, "f32" if io == "f32" else "bf16", "hT")


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("shape", FUSED_FWD)
def test_full_backward_fused(rb, shape, io):
    """Layer backward over several tiles, with h0 and dL/dh_T given."""
    B, L, D = shape
    f = dg.full_inputs(B, L, D, 4400 + B + L + D, io=io, a_range=(0.99, 0.9999), bias=True,
                       h0=True, grad=True, dhT=True)
    X, Wr, br, Wi, bi = (dev(a, io) for a in (f.x, f.Wr, f.br, f.Wi, f.bi))
    lam, h0 = dev32(f.lam), dev32(f.h0)
    h, _ = rb.bdlru_forward(X, Wr, br, Wi, bi, lam, h0)
    got = rb.bdlru_backward(X, Wr, br, Wi, bi, lam, h, dev(f.dh, io), h0, dev32(f.dhT))
    print(f"fused backward {shape} {io}: GPU done", flush=True)
    want = oracle.backward(f.x, f.Wr, f.br, f.Wi, f.bi, f.lam, f.dh, f.h0, f.dhT)
    for k in ("dx", "dWr", "dbr", "dWi", "dbi", "dlambda", "dh0"):
        assert_close(host(got[k]), want[k], io, k)


# (B, D): D % 8 == 0 runs the step fused with the projection (z in registers),
# with a partial channel block for D = 72; D = 130 takes the two-kernel path.
@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(50, 64), (300, 72), (129, 256), (7, 130)])
def test_full_step(rb, io, shape):
    B, D = shape
    f = dg.full_inputs(B, 1, D, 4100 + B + D, io=io, bias=True, h0=True)
    x = f.x[:, 0]
    got = rb.bdlru_step(dev(x, io), dev(f.Wr, io), dev(f.br, io), dev(f.Wi, io), dev(f.bi, io),
                        dev32(f.lam), dev32(f.h0))
    want = oracle.step(x, f.Wr, f.br, f.Wi, f.bi, f.lam, f.h0)
    assert_close(host(got), want, io, "h_next")


# bf16 with D in {64, 128, 192, 256} runs the step with the weights resident
# in registers: blocks of 16 rows handed out round-robin to persistent
# workgroups.  B = 12293 gives 769 blocks at D = 256 (an odd count for some
# workgroups, which ends on a half round) and a ragged last block; B = 5 is
# one partial block.
@pytest.mark.parametrize("shape,bias", [((5, 64), True), ((4111, 128), True),
                                        ((1000, 192), False), ((33, 256), True),
                                        ((12293, 256), True), ((40000, 64), False)])
def test_full_step_resident(rb, shape, bias):
    B, D = shape
    f = dg.full_inputs(B, 1, D, 4170 + B + D, io="bf16", bias=bias, h0=True)
    x = f.x[:, 0]
    br = dev(f.br, "bf16") if bias else None
    bi = dev(f.bi, "bf16") if bias else None
    got = rb.bdlru_step(dev(x, "bf16"), dev(f.Wr, "bf16"), br, dev(f.Wi, "bf16"), bi,
                        dev32(f.lam), dev32(f.h0))
    want = oracle.step(x, f.Wr, f.br if bias else None, f.Wi, f.bi if bias else None, f.lam,
                       f.h0)
    assert_close(host(got), want, "bf16", "h_next")


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_full_step_in_place(rb, io):
    """h_next may be h_prev; two steps in a row match two oracle steps."""
    import torch
    B, D = 200, 128
    f = dg.full_inputs(B, 2, D, 4150, io=io, bias=True, h0=True)
    W = [dev(a, io) for a in (f.Wr, f.br, f.Wi, f.bi)]
    lam = dev32(f.lam)
    h = dev32(f.h0)
    io_code = rb.io_code(torch.float32 if io == "f32" else torch.bfloat16)
    nws = rb.recblr_workspace_size(rb.OP_STEP, B, 1, D, io_code)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=h.device)
    want = f.h0.astype(np.float64)
    for t in range(2):
        xt = dev(np.ascontiguousarray(f.x[:, t]), io)
        st = rb.recblr_bdlru_step(xt.data_ptr(), W[0].data_ptr(), W[1].data_ptr(),
                                  W[2].data_ptr(), W[3].data_ptr(), lam.data_ptr(),
                                  h.data_ptr(), h.data_ptr(), B, D, io_code, ws.data_ptr(), nws,
                                  torch.cuda.current_stream().cuda_stream)
        assert st == 0, st
        want = oracle.step(f.x[:, t], f.Wr, f.br, f.Wi, f.bi, f.lam, want)
    assert_close(host(h), want, "f32" if io == "f32" else "bf16", "h after two in-place steps")


def test_full_forward_without_bias(rb):
    f = dg.full_inputs(2, 20, 64, 4200)
    X, Wr, Wi = dev(f.x), dev(f.Wr), dev(f.Wi)
    h, hT = rb.bdlru_forward(X, Wr, None, Wi, None, dev32(f.lam))
    oh, _ = oracle.forward(f.x, f.Wr, None, f.Wi, None, f.lam)
    assert_close(host(h), oh, "f32", "h")


# ------------------------------------------------------------------ efficiency-ablation scans

ABLATION_SHAPES = [(3, 200, 64), (2, 257, 128), (4, 100, 72), (1, 1, 8), (2, 64, 32),
                   (1, 1000, 16)]


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("shape", ABLATION_SHAPES)
@pytest.mark.parametrize("method", ["serial", "tree"])
def test_scan_methods(rb, method, shape, io):
    B, L, D = shape
    inp = dg.scan_inputs(B, L, D, 6000 + B + L + D, io=io)
    m = rb.SCAN_SERIAL if method == "serial" else rb.SCAN_TREE
    h = rb.scan_forward_method(m, dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io),
                               dev32(inp.lam))
    oh, _ = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam)
    assert_close(host(h), oh, io, f"{method} h")


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("shape", ABLATION_SHAPES)
@pytest.mark.parametrize("method", ["serial", "tree", "chunked"])
def test_scan_backward_methods(rb, method, shape, io):
    """Backward of the ablation's scans (zero initial state) against the oracle."""
    B, L, D = shape
    inp = dg.scan_inputs(B, L, D, 6200 + B + L + D, io=io, grad=True)
    m = {"serial": rb.SCAN_SERIAL, "tree": rb.SCAN_TREE, "chunked": rb.SCAN_CHUNKED}[method]
    X, ZR, ZI, lam = dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io), dev32(inp.lam)
    h = rb.scan_forward_method(m, X, ZR, ZI, lam)
    g = rb.scan_backward_method(m, X, ZR, ZI, lam, h, dev(inp.dh, io))
    want = oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh)
    for k in ("dx", "dzr", "dzi", "dlambda"):
        assert_close(host(g[k]), want[k], io, f"{method} {k}")


def test_tree_scan_sequence_padding(rb):
    """Sequence padding: inputs left-padded to a power of two with zero x
    (any z) give the unpadded result on the real positions (zero state)."""
    B, L, D, P = 3, 200, 64, 256
    inp = dg.scan_inputs(B, L, D, 6100)
    pad = dg.scan_inputs(B, P - L, D, 6101)
    x = np.concatenate([np.zeros_like(pad.x), inp.x], axis=1)
    zr = np.concatenate([pad.zr, inp.zr], axis=1)
    zi = np.concatenate([pad.zi, inp.zi], axis=1)
    h = rb.scan_forward_method(rb.SCAN_TREE, dev(x), dev(zr), dev(zi), dev32(inp.lam))
    oh, _ = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam)
    assert_close(host(h)[:, P - L:], oh, "f32", "tree h, sequence padding")


# ------------------------------------------------------------------ gated recurrent layer core
# D = 128 (fp32, bf16) and D = 256 (bf16) take the weights-resident fused
# kernel with the conv on load (look-back mode with few channel groups, chain
# mode with 256); other D % 64 == 0 shapes the tile kernel, the rest the
# unfused path.  The D = 128 / 256 cases with L below the conv's 3-row halo,
# a last tile of one row and K = 3 exercise the staged halo of the conv.
GATED_CASES = [((2, 300, 64), 4), ((1, 700, 128), 2), ((1, 513, 256), 1), ((8, 50, 64), 4),
               ((2, 300, 72), 3), ((3, 1, 64), 4), ((256, 70, 128), 4), ((2, 2, 128), 3),
               ((1, 65, 256), 4), ((4, 130, 128), 3), ((3, 1, 256), 2)]


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("case", GATED_CASES)
def test_gated_forward(rb, case, io):
    import torch
    (B, L, D), K = case
    f = dg.full_inputs(B, L, D, 8000 + B + L + D + K, io=io, a_range=(0.99, 0.9999), bias=True,
                       h0=True)
    rng = np.random.default_rng(8000 + L)
    hz = rng.standard_normal((B, L, D)).astype(np.float32)
    if io == "bf16":
        hz = dg.round_bf16(hz)
    w = (rng.standard_normal((D, K)) * 0.5).astype(np.float32)
    cb = (rng.standard_normal(D) * 0.1).astype(np.float32)
    y, h, hT = rb.gated_forward(dev(f.x, io), dev(hz, io), dev32(w), dev32(cb),
                                *(dev(a, io) for a in (f.Wr, f.br, f.Wi, f.bi)), dev32(f.lam),
                                dev32(f.h0))
    y2, h2, _ = rb.gated_forward(dev(f.x, io), dev(hz, io), dev32(w), None,
                                 *(dev(a, io) for a in (f.Wr, f.br, f.Wi, f.bi)), dev32(f.lam),
                                 keep_h=False)
    torch.cuda.synchronize()
    print(f"gated {case} {io}: GPU done", flush=True)
    oy, oh, ohT = oracle.gated_forward(f.x, hz, w, cb, f.Wr, f.br, f.Wi, f.bi, f.lam, f.h0)
    assert_close(host(y), oy, io, "y")
    assert_close(host(h), oh, io, "h")
    assert_close(host(hT), ohT, "f32" if io == "f32" else "bf16", "hT")
    oy2, _, _ = oracle.gated_forward(f.x, hz, w, None, f.Wr, f.br, f.Wi, f.bi, f.lam)
    assert h2 is None
    assert_close(host(y2), oy2, io, "y (no bias, no h0, h not kept)")


GATED_BWD_CASES = [((2, 300, 64), 4), ((1, 700, 128), 2), ((3, 130, 72), 3), ((8, 50, 64), 1),
                   ((2, 5, 8), 4), ((3, 1, 64), 4), ((2, 0, 64), 3)]


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("case", GATED_BWD_CASES)
def test_gated_backward(rb, case, io):
    """Every gradient of the gated layer core against the oracle's chain rule,
    with and without a conv bias / h0 / dhT."""
    import torch
    (B, L, D), K = case
    seed = 8100 + B + L + D + K
    f = dg.full_inputs(B, L, D, seed, io=io, a_range=(0.99, 0.9999), bias=True, h0=True,
                       grad=True, dhT=True)
    rng = np.random.default_rng(seed)
    hz = rng.standard_normal((B, L, D)).astype(np.float32)
    if io == "bf16":
        hz = dg.round_bf16(hz)
    w = (rng.standard_normal((D, K)) * 0.5).astype(np.float32)
    cb = (rng.standard_normal(D) * 0.1).astype(np.float32)
    args = [dev(f.Wr, io), dev(f.br, io), dev(f.Wi, io), dev(f.bi, io), dev32(f.lam)]
    HX, HZ, DY = dev(f.x, io), dev(hz, io), dev(f.dh, io)
    _, h, _ = rb.gated_forward(HX, HZ, dev32(w), dev32(cb), *args, dev32(f.h0))
    got = rb.gated_backward(HX, HZ, dev32(w), dev32(cb), *args, h, DY, dev32(f.h0),
                            dev32(f.dhT))
    _, h2, _ = rb.gated_forward(HX, HZ, dev32(w), None, *args)
    got2 = rb.gated_backward(HX, HZ, dev32(w), None, *args, h2, DY)
    torch.cuda.synchronize()
    print(f"gated backward {case} {io}: GPU done", flush=True)
    want = oracle.gated_backward(f.x, hz, w, cb, f.Wr, f.br, f.Wi, f.bi, f.lam, f.dh, f.h0,
                                 f.dhT)
    for k in ("dhx", "dhz", "dconv_w", "dconv_b", "dWr", "dbr", "dWi", "dbi", "dlambda", "dh0"):
        assert_close(host(got[k]), want[k], io, k)
    want2 = oracle.gated_backward(f.x, hz, w, None, f.Wr, f.br, f.Wi, f.bi, f.lam, f.dh)
    assert got2["dconv_b"] is None and got2["dh0"] is None
    for k in ("dhx", "dhz", "dconv_w", "dWr", "dlambda"):
        assert_close(host(got2[k]), want2[k], io, k + " (no bias, no h0)")


# ------------------------------------------------------------------ named workloads at full size
# Every element of every output is compared with the oracle (the oracle runs
# the whole batch); the error report of each output is printed.

@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_config_full_size(rb, name):
    import torch
    cfg = dg.CONFIGS[name]
    inp = dg.config_inputs(cfg, grad=True)
    io = cfg.io
    X, ZR, ZI, lam = dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io), dev32(inp.lam)
    h, hT = rb.bdlru_scan_forward(X, ZR, ZI, lam)
    g = rb.bdlru_scan_backward(X, ZR, ZI, lam, h, dev(inp.dh, io))
    torch.cuda.synchronize()
    print(f"config {name}: GPU done", flush=True)
    got = {"h": host(h), "hT": host(hT)}
    got.update({k: host(g[k]) for k in ("dx", "dzr", "dzi", "dh0", "dlambda")})
    del h, hT, g, X, ZR, ZI
    oh, ohT = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam)
    ob = oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh)
    ob.update(h=oh, hT=ohT)
    for k in ("h", "hT", "dx", "dzr", "dzi", "dh0", "dlambda"):
        report(f"scan {name} {k}", got[k], ob[k])
        assert_close(got[k], ob[k], io, f"{name} {k}")


def test_config_decode_full_api(rb):
    """The decode workload through the entry point with gate weights (fused path)."""
    cfg = dg.CONFIGS["c5dec"]
    f = dg.full_inputs(cfg.B, 1, cfg.D, cfg.seed + 100, io=cfg.io, a_range=cfg.a_range,
                       bias=True, h0=True)
    x = f.x[:, 0]
    got = rb.bdlru_step(dev(x, cfg.io), dev(f.Wr, cfg.io), dev(f.br, cfg.io), dev(f.Wi, cfg.io),
                        dev(f.bi, cfg.io), dev32(f.lam), dev32(f.h0))
    want = oracle.step(x, f.Wr, f.br, f.Wi, f.bi, f.lam, f.h0)
    report("decode full API h_next", host(got), want)
    assert_close(host(got), want, cfg.io, "decode h_next (full API)")


def test_config_decode_full_size(rb):
    cfg = dg.CONFIGS["c5dec"]
    inp = dg.step_inputs(cfg.B, cfg.D, cfg.seed, io=cfg.io, a_range=cfg.a_range)
    got = rb.bdlru_scan_step(dev(inp.x, cfg.io), dev(inp.zr, cfg.io), dev(inp.zi, cfg.io),
                             dev32(inp.lam), dev32(inp.h0))
    want = oracle.scan_step(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
    report("decode h_next", host(got), want)
    assert_close(host(got), want, cfg.io, "decode h_next")


@pytest.mark.parametrize("name", ["c3", "c4", "c5"])
def test_config_full_api(rb, name):
    """Entry points with gate parameters at the workload's full size, every
    element of h, hT and dx and every weight gradient against the oracle over
    the whole batch."""
    import torch
    cfg = dg.CONFIGS[name]
    io = cfg.io
    f = dg.full_inputs(cfg.B, cfg.L, cfg.D, cfg.seed + 100, io=io, a_range=cfg.a_range,
                       bias=True, grad=True)
    X, Wr, br, Wi, bi = (dev(a, io) for a in (f.x, f.Wr, f.br, f.Wi, f.bi))
    lam = dev32(f.lam)
    h, hT = rb.bdlru_forward(X, Wr, br, Wi, bi, lam)
    g = rb.bdlru_backward(X, Wr, br, Wi, bi, lam, h, dev(f.dh, io))
    torch.cuda.synchronize()
    print(f"full API {name}: GPU done", flush=True)
    got = {"h": host(h), "hT": host(hT)}
    got.update({k: host(g[k]) for k in ("dx", "dWr", "dbr", "dWi", "dbi", "dlambda", "dh0")})
    del h, hT, g, X
    oh, ohT = oracle.forward(f.x, f.Wr, f.br, f.Wi, f.bi, f.lam)
    want = oracle.backward(f.x, f.Wr, f.br, f.Wi, f.bi, f.lam, f.dh)
    want.update(h=oh, hT=ohT)
    for k in ("h", "hT", "dx", "dWr", "dbr", "dWi", "dbi", "dlambda", "dh0"):
        r = report(f"full API {name} {k}", got[k], want[k])
        assert_close(got[k], want[k], io, f"{name} {k}")
        if io == "f32":
            # The fp32 projections run on bf16 matrix cores with a 3-term
            # split (each product exact to about 3 * 2^-17): keep a 2x margin
            # under the 1e-4 bar at the full workloads.
            assert r["floored"] <= 5e-5, f"{name} {k}: fp32 projection margin {r['floored']:.2e}"


# ------------------------------------------------------------------ kernel modes
# Few channel groups and long sequences run the look-back kernels (forward:
# under 256 groups of 64 channels, backward: under 1024); many channel groups
# run the chain kernels.  Forward chain lanes carry 1, 2 or 4 channels
# depending on D, the I/O type and pointer alignment.
MODE_CASES = [
    ((1, 5000, 64), "f32"),    # look-back, one channel group
    ((2, 3000, 256), "bf16"),  # look-back, 8 groups
    ((1, 2000, 3), "f32"),     # look-back, mostly idle lanes
    ((3, 1000, 40), "f32"),    # look-back, partially idle group
    ((64, 300, 512), "f32"),   # chain forward, 2 channels per lane; look-back backward
    ((64, 130, 1024), "bf16"), # chain, 4 channels per lane forward; chain backward
    ((11000, 70, 3), "f32"),   # chain, 1 channel per lane, ragged last group
]


@pytest.mark.parametrize("shape,io", MODE_CASES)
def test_kernel_modes(rb, shape, io):
    B, L, D = shape
    inp = dg.scan_inputs(B, L, D, 5000 + B + L + D, io=io, h0=True, grad=True, dhT=True)
    X, ZR, ZI = dev(inp.x, io), dev(inp.zr, io), dev(inp.zi, io)
    lam, h0 = dev32(inp.lam), dev32(inp.h0)
    h, hT = rb.bdlru_scan_forward(X, ZR, ZI, lam, h0)
    got = rb.bdlru_scan_backward(X, ZR, ZI, lam, h, dev(inp.dh, io), h0, dev32(inp.dhT))
    print(f"mode case {shape} {io}: GPU done", flush=True)
    oh, ohT = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
    assert_close(host(h), oh, io, "h")
    assert_close(host(hT), ohT, "f32", "hT")
    want = oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh, inp.h0, inp.dhT)
    for k in ("dx", "dzr", "dzi", "dlambda"):
        assert_close(host(got[k]), want[k], io, k)
    assert_close(host(got["dh0"]), want["dh0"], "f32", "dh0")


@pytest.mark.parametrize("shape,io", [((2, 700, 64), "f32"), ((64, 300, 512), "f32"),
                                      ((2, 1000, 256), "bf16"), ((300, 90, 64), "bf16")])
def test_timed_scans(rb, shape, io):
    """The measurement entry points compute bit for bit what the plain ones do,
    and the event pair they record brackets a positive duration."""
    import torch
    B, L, D = shape
    inp = dg.scan_inputs(B, L, D, 5200 + L, io=io, h0=True, grad=True)
    X, ZR, ZI, DH = (dev(a, io) for a in (inp.x, inp.zr, inp.zi, inp.dh))
    lam, h0 = dev32(inp.lam), dev32(inp.h0)
    code = rb.io_code(X.dtype)
    p = lambda t: t.data_ptr()
    s = torch.cuda.current_stream().cuda_stream
    nf = rb.recblr_workspace_size(rb.OP_SCAN_FORWARD, B, L, D, code)
    nb = rb.recblr_workspace_size(rb.OP_SCAN_BACKWARD, B, L, D, code)
    wsf = torch.empty(max(nf, 1), dtype=torch.uint8, device=X.device)
    wsb = torch.empty(max(nb, 1), dtype=torch.uint8, device=X.device)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev:
        e.record()
    outs = []
    for timed in (False, True):
        h, dx, dzr, dzi = (torch.empty_like(X) for _ in range(4))
        hT, dh0 = (torch.empty((B, D), dtype=torch.float32, device=X.device) for _ in range(2))
        dl = torch.empty(D, dtype=torch.float32, device=X.device)
        fa = (p(X), p(ZR), p(ZI), p(lam), p(h0), p(h), p(hT), B, L, D, code, p(wsf), nf, s)
        ba = (p(X), p(ZR), p(ZI), p(lam), p(h0), p(h), p(DH), None, p(dx), p(dzr), p(dzi),
              p(dl), p(dh0), B, L, D, code, p(wsb), nb, s)
        if timed:
            assert rb.recblr_bdlru_scan_forward_timed(*fa, ev[0].cuda_event, ev[1].cuda_event) == 0
            assert rb.recblr_bdlru_scan_backward_timed(*ba, ev[2].cuda_event, ev[3].cuda_event) == 0
        else:
            assert rb.recblr_bdlru_scan_forward(*fa) == 0
            assert rb.recblr_bdlru_scan_backward(*ba) == 0
        torch.cuda.synchronize()
        outs.append([host(t) for t in (h, hT, dx, dzr, dzi, dl, dh0)])
    print(f"timed scans {shape} {io}: GPU done", flush=True)
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
    assert ev[0].elapsed_time(ev[1]) > 0 and ev[2].elapsed_time(ev[3]) > 0


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_misaligned_pointers(rb, io):
    """Tensors that start one element past an aligned address take the 1-channel lanes."""
    import torch
    B, L, D = 2, 700, 64
    inp = dg.scan_inputs(B, L, D, 5100, io=io, h0=True, grad=True)
    n = B * L * D

    def shifted(a, iot):
        t = dev(a.reshape(-1), iot)
        buf = torch.empty(n + 1, dtype=t.dtype, device=t.device)
        buf[1:] = t
        return buf[1:].view(B, L, D)

    X, ZR, ZI, DH = (shifted(a, io) for a in (inp.x, inp.zr, inp.zi, inp.dh))
    assert X.data_ptr() % 8 != 0
    lam, h0 = dev32(inp.lam), dev32(inp.h0)
    h, hT = rb.bdlru_scan_forward(X, ZR, ZI, lam, h0)
    got = rb.bdlru_scan_backward(X, ZR, ZI, lam, h, DH, h0)
    oh, ohT = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
    assert_close(host(h), oh, io, "h")
    want = oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh, inp.h0)
    for k in ("dx", "dzr", "dzi", "dlambda"):
        assert_close(host(got[k]), want[k], io, k)


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_full_backward_misaligned_h(rb, io):
    """The layer backward with h (the saved forward output) one element past a
    16-byte boundary: the fused backward stages h with 16-byte loads, so such
    a call must take the path through the separate projection kernels, and
    still match the oracle."""
    import torch
    B, L, D = 2, 300, 128
    f = dg.full_inputs(B, L, D, 5300, io=io, a_range=(0.99, 0.9999), bias=True, h0=True,
                       grad=True, dhT=True)
    X, Wr, br, Wi, bi = (dev(a, io) for a in (f.x, f.Wr, f.br, f.Wi, f.bi))
    lam, h0 = dev32(f.lam), dev32(f.h0)
    h, _ = rb.bdlru_forward(X, Wr, br, Wi, bi, lam, h0)
    buf = torch.empty(h.numel() + 1, dtype=h.dtype, device=h.device)
    buf[1:] = h.reshape(-1)
    hs = buf[1:].view(B, L, D)
    assert hs.data_ptr() % 16 != 0
    got = rb.bdlru_backward(X, Wr, br, Wi, bi, lam, hs, dev(f.dh, io), h0, dev32(f.dhT))
    ref = rb.bdlru_backward(X, Wr, br, Wi, bi, lam, h, dev(f.dh, io), h0, dev32(f.dhT))
    torch.cuda.synchronize()
    want = oracle.backward(f.x, f.Wr, f.br, f.Wi, f.bi, f.lam, f.dh, f.h0, f.dhT)
    for k in ("dx", "dWr", "dbr", "dWi", "dbi", "dlambda", "dh0"):
        assert_close(host(got[k]), want[k], io, k)
        assert_close(host(ref[k]), want[k], io, k + " (aligned h)")


def test_explicit_stream(rb):
    """Wrappers called with a stream other than torch's current one allocate
    their workspace and outputs on that stream; results match the oracle."""
    import torch
    inp = dg.scan_inputs(2, 1500, 64, 5400, h0=True, grad=True, dhT=True)
    s = torch.cuda.Stream()
    X, ZR, ZI, DH = (dev(a) for a in (inp.x, inp.zr, inp.zi, inp.dh))
    lam, h0, dhT = dev32(inp.lam), dev32(inp.h0), dev32(inp.dhT)
    s.wait_stream(torch.cuda.current_stream())
    outs = []
    for _ in range(3):  # repeated calls: a reused workspace must not be handed out early
        h, hT = rb.bdlru_scan_forward(X, ZR, ZI, lam, h0, stream=s)
        g = rb.bdlru_scan_backward(X, ZR, ZI, lam, h, DH, h0, dhT, stream=s)
        # an allocation on the current stream right after the call
        junk = torch.full((1 << 20,), 7.0, device=X.device)
        outs.append((h, hT, g, junk))
    s.synchronize()
    torch.cuda.synchronize()
    oh, ohT = oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam, inp.h0)
    want = oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh, inp.h0, inp.dhT)
    for h, hT, g, _ in outs:
        assert_close(host(h), oh, "f32", "h")
        assert_close(host(hT), ohT, "f32", "hT")
        for k in ("dx", "dzr", "dzi", "dlambda", "dh0"):
            assert_close(host(g[k]), want[k], "f32", k)


@pytest.mark.parametrize("shape,io", [((1, 5000, 64), "f32"), ((2, 3000, 256), "bf16"),
                                      ((64, 300, 512), "f32"), ((11000, 70, 3), "f32")])
def test_workspace_status_word(rb, shape, io):
    """The status word at byte 4 of the scan workspaces (set when a bounded
    look-back wait runs out) is cleared by every call, also from a workspace
    full of 0xFF, and stays 0 in normal operation."""
    import torch
    B, L, D = shape
    inp = dg.scan_inputs(B, L, D, 5500 + L, io=io, grad=True)
    X, ZR, ZI, DH = (dev(a, io) for a in (inp.x, inp.zr, inp.zi, inp.dh))
    lam = dev32(inp.lam)
    code = rb.io_code(X.dtype)
    s = torch.cuda.current_stream().cuda_stream
    p = lambda t: t.data_ptr()
    h = torch.empty_like(X)
    nf = rb.recblr_workspace_size(rb.OP_SCAN_FORWARD, B, L, D, code)
    nb = rb.recblr_workspace_size(rb.OP_SCAN_BACKWARD, B, L, D, code)
    wsf = torch.full((max(nf, 8),), 0xFF, dtype=torch.uint8, device=X.device)
    wsb = torch.full((max(nb, 8),), 0xFF, dtype=torch.uint8, device=X.device)
    assert rb.recblr_bdlru_scan_forward(p(X), p(ZR), p(ZI), p(lam), None, p(h), None, B, L, D,
                                        code, p(wsf) if nf else None, nf, s) == 0
    outs = [torch.empty_like(X) for _ in range(3)]
    dl = torch.empty(D, dtype=torch.float32, device=X.device)
    assert rb.recblr_bdlru_scan_backward(p(X), p(ZR), p(ZI), p(lam), None, p(h), p(DH), None,
                                         *(p(o) for o in outs), p(dl), None, B, L, D, code,
                                         p(wsb), nb, s) == 0
    torch.cuda.synchronize()
    assert nb > 0
    assert int(wsb[4:8].view(torch.int32).item()) == 0
    if nf:
        assert int(wsf[4:8].view(torch.int32).item()) == 0
