"""Guard bands around every output of every librecblr.so entry point.

Each output (and the workspace) is placed in the middle of a larger device
buffer whose bytes are all 0xFF: 4 KiB of poison before it and 4 KiB after
its last byte (so the output keeps the 256-byte alignment of a plain
allocation).  After the call the poison on both sides must be untouched, and
the output itself must equal, bit for bit, what the same call writes into a
plain allocation (the other parity tests check those against the fp64
oracle).  0xFF bytes read as NaN in fp32 and in bf16, so an element the call
failed to write also shows up.  Shapes cover ragged tiles (L not a multiple
of the 128-step tiles, B*D not a multiple of 64 channels, idle lanes), both
kernel modes, the fused paths and the named workloads at full size.
"""
import numpy as np
import pytest

from helpers import dev, dev32
from paper_2406_12580_amd import datagen as dg

pytestmark = pytest.mark.gpu

GUARD = 4096
POISON = 0xFF


@pytest.fixture(scope="module")
def rb():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2406_12580_amd import recblr
    return recblr


class Guarded:
    """A tensor of `shape` and `dtype` with poisoned bytes on both sides."""

    def __init__(self, shape, dtype):
        import torch
        esz = torch.empty((), dtype=dtype).element_size()
        self.n = int(np.prod(shape)) * esz
        self.buf = torch.full((GUARD + self.n + GUARD,), POISON, dtype=torch.uint8,
                              device="cuda")
        self.t = self.buf[GUARD:GUARD + self.n].view(dtype).view(shape)

    @property
    def ptr(self):
        return self.t.data_ptr()

    def check(self, name):
        head = self.buf[:GUARD].cpu().numpy()
        tail = self.buf[GUARD + self.n:].cpu().numpy()
        assert (head == POISON).all(), f"{name}: {int((head != POISON).sum())} bytes written before"
        assert (tail == POISON).all(), f"{name}: {int((tail != POISON).sum())} bytes written after"


def _ws(rb, op, B, L, D, io):
    import torch
    n = rb.recblr_workspace_size(op, B, L, D, io)
    return Guarded((max(n, 1),), torch.uint8), n


def _same(got, want, name):
    import torch
    a = got.detach().contiguous().view(torch.uint8).cpu().numpy()
    b = want.detach().contiguous().view(torch.uint8).cpu().numpy()
    assert a.shape == b.shape, name
    assert np.array_equal(a, b), f"{name}: differs from the unguarded call"


def _stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def _sync():
    import torch
    torch.cuda.synchronize()


# ------------------------------------------------------------------ scan level

def _guard_scan(rb, inp, with_state):
    import torch
    io = inp.io
    X, ZR, ZI, DH = (dev(a, io) for a in (inp.x, inp.zr, inp.zi, inp.dh))
    lam = dev32(inp.lam)
    h0 = dev32(inp.h0) if with_state else None
    dhT = dev32(inp.dhT) if with_state else None
    B, L, D = inp.x.shape
    code = rb.io_code(X.dtype)
    f32 = torch.float32
    h, hT = Guarded((B, L, D), X.dtype), Guarded((B, D), f32)
    wsf, nf = _ws(rb, rb.OP_SCAN_FORWARD, B, L, D, code)
    p = lambda t: None if t is None else t.data_ptr()
    st = rb.recblr_bdlru_scan_forward(p(X), p(ZR), p(ZI), p(lam), p(h0), h.ptr, hT.ptr, B, L, D,
                                      code, wsf.ptr, nf, _stream())
    assert st == 0, st
    outs = {k: Guarded((B, L, D), X.dtype) for k in ("dx", "dzr", "dzi")}
    outs["dlambda"], outs["dh0"] = Guarded((D,), f32), Guarded((B, D), f32)
    wsb, nb = _ws(rb, rb.OP_SCAN_BACKWARD, B, L, D, code)
    st = rb.recblr_bdlru_scan_backward(p(X), p(ZR), p(ZI), p(lam), p(h0), h.ptr, p(DH), p(dhT),
                                       outs["dx"].ptr, outs["dzr"].ptr, outs["dzi"].ptr,
                                       outs["dlambda"].ptr, outs["dh0"].ptr, B, L, D, code,
                                       wsb.ptr, nb, _stream())
    assert st == 0, st
    rh, rhT = rb.bdlru_scan_forward(X, ZR, ZI, lam, h0)
    ref = rb.bdlru_scan_backward(X, ZR, ZI, lam, rh, DH, h0, dhT)
    _sync()
    print(f"guard scan {inp.x.shape} {io}: GPU done", flush=True)
    for g, name in ((h, "h"), (hT, "hT"), (wsf, "forward workspace"),
                    (wsb, "backward workspace"), *((outs[k], k) for k in outs)):
        g.check(name)
    _same(h.t, rh, "h")
    _same(hT.t, rhT, "hT")
    for k in outs:
        _same(outs[k].t, ref[k], k)


# (B, L, D): idle lanes (B*D % 64 != 0), ragged tiles along L, look-back and
# chain modes, VEC = 2 / 4 chain lanes.
SCAN_CASES = [((3, 777, 100), "f32"), ((3, 777, 100), "bf16"), ((1, 5000, 64), "f32"),
              ((2, 3000, 256), "bf16"), ((1, 2000, 3), "f32"), ((64, 300, 512), "f32"),
              ((64, 130, 1024), "bf16"), ((11000, 70, 3), "f32"), ((2, 1, 64), "bf16")]


@pytest.mark.parametrize("shape,io", SCAN_CASES)
def test_guard_scan(rb, shape, io):
    B, L, D = shape
    inp = dg.scan_inputs(B, L, D, 9000 + B + L + D, io=io, h0=True, grad=True, dhT=True)
    _guard_scan(rb, inp, True)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_guard_scan_configs(rb, name):
    cfg = dg.CONFIGS[name]
    _guard_scan(rb, dg.config_inputs(cfg, grad=True), False)


# ------------------------------------------------------------------ entry points with weights

def _guard_full(rb, f, with_state):
    import torch
    io = f.io
    X, Wr, br, Wi, bi, DH = (dev(a, io) for a in (f.x, f.Wr, f.br, f.Wi, f.bi, f.dh))
    lam = dev32(f.lam)
    h0 = dev32(f.h0) if with_state else None
    dhT = dev32(f.dhT) if with_state else None
    B, L, D = f.x.shape
    code = rb.io_code(X.dtype)
    f32 = torch.float32
    p = lambda t: None if t is None else t.data_ptr()
    h, hT = Guarded((B, L, D), X.dtype), Guarded((B, D), f32)
    wsf, nf = _ws(rb, rb.OP_FORWARD, B, L, D, code)
    st = rb.recblr_bdlru_forward(p(X), p(Wr), p(br), p(Wi), p(bi), p(lam), p(h0), h.ptr, hT.ptr,
                                 B, L, D, code, wsf.ptr, nf, _stream())
    assert st == 0, st
    outs = {"dx": Guarded((B, L, D), X.dtype), "dWr": Guarded((D, D), f32),
            "dbr": Guarded((D,), f32), "dWi": Guarded((D, D), f32), "dbi": Guarded((D,), f32),
            "dlambda": Guarded((D,), f32), "dh0": Guarded((B, D), f32)}
    wsb, nb = _ws(rb, rb.OP_BACKWARD, B, L, D, code)
    st = rb.recblr_bdlru_backward(p(X), p(Wr), p(br), p(Wi), p(bi), p(lam), p(h0), h.ptr, p(DH),
                                  p(dhT), outs["dx"].ptr, outs["dWr"].ptr, outs["dbr"].ptr,
                                  outs["dWi"].ptr, outs["dbi"].ptr, outs["dlambda"].ptr,
                                  outs["dh0"].ptr, B, L, D, code, wsb.ptr, nb, _stream())
    assert st == 0, st
    rh, rhT = rb.bdlru_forward(X, Wr, br, Wi, bi, lam, h0)
    ref = rb.bdlru_backward(X, Wr, br, Wi, bi, lam, rh, DH, h0, dhT)
    _sync()
    print(f"guard full {f.x.shape} {io}: GPU done", flush=True)
    for g, name in ((h, "h"), (hT, "hT"), (wsf, "forward workspace"),
                    (wsb, "backward workspace"), *((outs[k], k) for k in outs)):
        g.check(name)
    _same(h.t, rh, "h")
    _same(hT.t, rhT, "hT")
    for k in outs:
        _same(outs[k].t, ref[k], k)


# D % 64 == 0 with L not a multiple of 128 (fused tiles with a ragged last
# one), D = 72 / 130 (separate projection kernels, partial channel groups).
FULL_CASES = [((3, 700, 128), "f32"), ((2, 257, 192), "bf16"), ((1, 1000, 64), "bf16"),
              ((2, 300, 72), "f32"), ((3, 70, 130), "bf16")]


@pytest.mark.parametrize("shape,io", FULL_CASES)
def test_guard_full(rb, shape, io):
    B, L, D = shape
    f = dg.full_inputs(B, L, D, 9100 + B + L + D, io=io, a_range=(0.99, 0.9999), bias=True,
                       h0=True, grad=True, dhT=True)
    _guard_full(rb, f, True)


@pytest.mark.parametrize("name", ["c3", "c4", "c5"])
def test_guard_full_configs(rb, name):
    cfg = dg.CONFIGS[name]
    f = dg.full_inputs(cfg.B, cfg.L, cfg.D, cfg.seed + 100, io=cfg.io, a_range=cfg.a_range,
                       bias=True, grad=True)
    _guard_full(rb, f, False)


# ------------------------------------------------------------------ decode steps

@pytest.mark.parametrize("shape,io", [((65536, 256), "bf16"), ((12293, 256), "bf16"),
                                      ((300, 72), "f32"), ((7, 130), "bf16"),
                                      ((33, 64), "f32")])
def test_guard_steps(rb, shape, io):
    import torch
    B, D = shape
    f = dg.full_inputs(B, 1, D, 9200 + B + D, io=io, bias=True, h0=True)
    si = dg.step_inputs(B, D, 9300 + B + D, io=io)
    x = dev(np.ascontiguousarray(f.x[:, 0]), io)
    Wr, br, Wi, bi = (dev(a, io) for a in (f.Wr, f.br, f.Wi, f.bi))
    lam, hp = dev32(f.lam), dev32(f.h0)
    code = rb.io_code(x.dtype)
    hn = Guarded((B, D), torch.float32)
    ws, nws = _ws(rb, rb.OP_STEP, B, 1, D, code)
    st = rb.recblr_bdlru_step(x.data_ptr(), Wr.data_ptr(), br.data_ptr(), Wi.data_ptr(),
                              bi.data_ptr(), lam.data_ptr(), hp.data_ptr(), hn.ptr, B, D, code,
                              ws.ptr, nws, _stream())
    assert st == 0, st
    sx, szr, szi = (dev(a, io) for a in (si.x, si.zr, si.zi))
    slam, shp = dev32(si.lam), dev32(si.h0)
    hs = Guarded((B, D), torch.float32)
    st = rb.recblr_bdlru_scan_step(sx.data_ptr(), szr.data_ptr(), szi.data_ptr(),
                                   slam.data_ptr(), shp.data_ptr(), hs.ptr, B, D, code,
                                   _stream())
    assert st == 0, st
    ref = rb.bdlru_step(x, Wr, br, Wi, bi, lam, hp)
    ref_s = rb.bdlru_scan_step(sx, szr, szi, slam, shp)
    _sync()
    print(f"guard steps {shape} {io}: GPU done", flush=True)
    for g, name in ((hn, "h_next"), (ws, "step workspace"), (hs, "scan step h_next")):
        g.check(name)
    _same(hn.t, ref, "h_next")
    _same(hs.t, ref_s, "scan step h_next")


# ------------------------------------------------------------------ gated layer core

@pytest.mark.parametrize("shape,io,K", [((2, 300, 64), "bf16", 4), ((1, 700, 128), "f32", 2),
                                        ((3, 130, 72), "f32", 3), ((16, 4000, 256), "bf16", 4)])
def test_guard_gated(rb, shape, io, K):
    import torch
    B, L, D = shape
    seed = 9400 + B + L + D
    f = dg.full_inputs(B, L, D, seed, io=io, a_range=(0.99, 0.9999), bias=True, h0=True,
                       grad=True, dhT=True)
    rng = np.random.default_rng(seed)
    hz = rng.standard_normal((B, L, D)).astype(np.float32)
    w = (rng.standard_normal((D, K)) * 0.5).astype(np.float32)
    cb = (rng.standard_normal(D) * 0.1).astype(np.float32)
    HX, HZ, DY = dev(f.x, io), dev(hz, io), dev(f.dh, io)
    W4, CB, lam, h0, dhT = dev32(w), dev32(cb), dev32(f.lam), dev32(f.h0), dev32(f.dhT)
    Wr, br, Wi, bi = (dev(a, io) for a in (f.Wr, f.br, f.Wi, f.bi))
    code = rb.io_code(HX.dtype)
    f32 = torch.float32
    p = lambda t: t.data_ptr()
    y, h, hT = Guarded((B, L, D), HX.dtype), Guarded((B, L, D), HX.dtype), Guarded((B, D), f32)
    wsf, nf = _ws(rb, rb.OP_GATED_FORWARD, B, L, D, code)
    st = rb.recblr_gated_forward(p(HX), p(HZ), p(W4), p(CB), K, p(Wr), p(br), p(Wi), p(bi),
                                 p(lam), p(h0), y.ptr, h.ptr, hT.ptr, B, L, D, code, wsf.ptr, nf,
                                 _stream())
    assert st == 0, st
    outs = {"dhx": Guarded((B, L, D), HX.dtype), "dhz": Guarded((B, L, D), HX.dtype),
            "dconv_w": Guarded((D, K), f32), "dconv_b": Guarded((D,), f32),
            "dWr": Guarded((D, D), f32), "dbr": Guarded((D,), f32), "dWi": Guarded((D, D), f32),
            "dbi": Guarded((D,), f32), "dlambda": Guarded((D,), f32),
            "dh0": Guarded((B, D), f32)}
    wsb, nb = _ws(rb, rb.OP_GATED_BACKWARD, B, L, D, code)
    o = {k: v.ptr for k, v in outs.items()}
    st = rb.recblr_gated_backward(p(HX), p(HZ), p(W4), p(CB), K, p(Wr), p(br), p(Wi), p(bi),
                                  p(lam), p(h0), h.ptr, p(DY), p(dhT), o["dhx"], o["dhz"],
                                  o["dconv_w"], o["dconv_b"], o["dWr"], o["dbr"], o["dWi"],
                                  o["dbi"], o["dlambda"], o["dh0"], B, L, D, code, wsb.ptr, nb,
                                  _stream())
    assert st == 0, st
    ry, rh, rhT = rb.gated_forward(HX, HZ, W4, CB, Wr, br, Wi, bi, lam, h0)
    ref = rb.gated_backward(HX, HZ, W4, CB, Wr, br, Wi, bi, lam, rh, DY, h0, dhT)
    _sync()
    print(f"guard gated {shape} {io} K={K}: GPU done", flush=True)
    for g, name in ((y, "y"), (h, "h"), (hT, "hT"), (wsf, "forward workspace"),
                    (wsb, "backward workspace"), *((outs[k], k) for k in outs)):
        g.check(name)
    _same(y.t, ry, "y")
    _same(h.t, rh, "h")
    _same(hT.t, rhT, "hT")
    for k in outs:
        _same(outs[k].t, ref[k], k)


# ------------------------------------------------------------------ diagnostic entry points

@pytest.mark.parametrize("shape,io", [((3, 200, 64), "f32"), ((4, 100, 72), "bf16"),
                                      ((1, 1000, 16), "f32")])
def test_guard_methods(rb, shape, io):
    import torch
    B, L, D = shape
    inp = dg.scan_inputs(B, L, D, 9500 + B + L + D, io=io, grad=True)
    X, ZR, ZI, DH = (dev(a, io) for a in (inp.x, inp.zr, inp.zi, inp.dh))
    lam = dev32(inp.lam)
    code = rb.io_code(X.dtype)
    p = lambda t: t.data_ptr()
    for m in (rb.SCAN_SERIAL, rb.SCAN_TREE, rb.SCAN_CHUNKED):
        h = Guarded((B, L, D), X.dtype)
        wsf, nf = _ws(rb, rb.OP_SCAN_FORWARD, B, L, D, code)
        st = rb.recblr_scan_forward_method(m, p(X), p(ZR), p(ZI), p(lam), h.ptr, B, L, D, code,
                                           wsf.ptr, nf, _stream())
        assert st == 0, st
        outs = {k: Guarded((B, L, D), X.dtype) for k in ("dx", "dzr", "dzi")}
        outs["dlambda"] = Guarded((D,), torch.float32)
        wsb, nb = _ws(rb, rb.OP_SCAN_BACKWARD_METHOD, B, L, D, code)
        st = rb.recblr_scan_backward_method(m, p(X), p(ZR), p(ZI), p(lam), h.ptr, p(DH),
                                            outs["dx"].ptr, outs["dzr"].ptr, outs["dzi"].ptr,
                                            outs["dlambda"].ptr, B, L, D, code, wsb.ptr, nb,
                                            _stream())
        assert st == 0, st
        rh = rb.scan_forward_method(m, X, ZR, ZI, lam)
        ref = rb.scan_backward_method(m, X, ZR, ZI, lam, rh, DH)
        _sync()
        for g, name in ((h, "h"), (wsf, "forward workspace"), (wsb, "backward workspace"),
                        *((outs[k], k) for k in outs)):
            g.check(f"method {m} {name}")
        _same(h.t, rh, f"method {m} h")
        for k in outs:
            _same(outs[k].t, ref[k], f"method {m} {k}")
    print(f"guard methods {shape} {io}: GPU done", flush=True)


def test_guard_linear_scan(rb):
    import torch
    B, L, D = 5, 333, 70
    rng = np.random.Generator(np.random.PCG64(9600))
    a = dev32(rng.uniform(0, 1, (B, L, D)).astype(np.float32))
    u = dev32(rng.standard_normal((B, L, D), dtype=np.float32))
    h0 = dev32(rng.standard_normal((B, D), dtype=np.float32))
    h, hT = Guarded((B, L, D), torch.float32), Guarded((B, D), torch.float32)
    st = rb.recblr_linear_scan_forward(a.data_ptr(), u.data_ptr(), h0.data_ptr(), h.ptr, hT.ptr,
                                       B, L, D, _stream())
    assert st == 0, st
    rh, rhT = rb.linear_scan_forward(a, u, h0)
    _sync()
    h.check("h")
    hT.check("hT")
    _same(h.t, rh, "h")
    _same(hT.t, rhT, "hT")


def test_guard_model_step(rb):
    """The model step's gradients and loss (with dropout and left-padded rows,
    so the mask and dropout-gradient regions of the workspace are used), and
    Adam's in-place updates."""
    import ctypes
    import torch
    dims = dg.ModelDims(B=64, T=130, D=64, E=2, V=500, layers=2, K=4)
    named = dg.model_params(dims, 9700)
    ids, targets = dg.model_batch(dims, 9701, min_len=10, pad_id=0)
    opts = rb.ModelStepOpts(0.3, 0, 77, 5)
    rd = rb.model_dims(dims.B, dims.T, dims.D, dims.E, dims.V, dims.layers, dims.K, dims.eps)
    offs = rb.model_param_offsets(rd)
    n = rb.recblr_model_param_count(rd)
    flat = np.zeros(n, dtype=np.float32)
    for (name, arr), o in zip(named.items(), offs):
        flat[o:o + arr.size] = arr.ravel()
    P = torch.from_numpy(flat).cuda()
    I, Tg = torch.from_numpy(ids).cuda(), torch.from_numpy(targets).cuda()
    step = rb.ModelStep(rd)
    G, loss = Guarded((n,), torch.float32), Guarded((1,), torch.float32)
    nws = rb.recblr_model_workspace_size(ctypes.byref(rd))
    ws = Guarded((nws,), torch.uint8)
    st = rb.recblr_model_train_step(ctypes.byref(rd), ctypes.byref(opts), P.data_ptr(),
                                    I.data_ptr(), Tg.data_ptr(), G.ptr, loss.ptr, ws.ptr, nws,
                                    step.blas, _stream())
    assert st == 0, st
    rloss, rG = step.train_step(P, I, Tg, dropout=0.3, seed=77, offset=5, pad_id=0)
    # Adam in place on guarded copies of the parameters and moments.
    params, m1, m2 = (Guarded((n,), torch.float32) for _ in range(3))
    params.t.copy_(P)
    m1.t.zero_()
    m2.t.zero_()
    st = rb.recblr_adam_update(params.ptr, rG.data_ptr(), m1.ptr, m2.ptr, n, 1, 1e-3, 0.9, 0.999,
                               1e-8, _stream())
    assert st == 0, st
    rp, rm1, rm2 = P.clone(), torch.zeros_like(P), torch.zeros_like(P)
    rb.adam_update(rp, rG, rm1, rm2, 1)
    _sync()
    print("guard model step: GPU done", flush=True)
    for g, name in ((G, "grads"), (loss, "loss"), (ws, "model workspace"), (params, "params"),
                    (m1, "m1"), (m2, "m2")):
        g.check(name)
    _same(G.t, rG, "grads")
    _same(loss.t, rloss, "loss")
    _same(params.t, rp, "params")
    _same(m1.t, rm1, "m1")
    _same(m2.t, rm2, "m2")
    step.close()
