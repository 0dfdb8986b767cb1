"""Host-only checks of the C ABI (no GPU needed).

The library must load and export every entry point include/recblr.h declares,
and every validation error must be reported before anything reaches the GPU.
Pointers here are fake addresses: every call below is rejected by host-side
validation, so no HIP call is made.
"""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "recblr.h")


@pytest.fixture(scope="module")
def rb():
    from paper_2406_12580_amd import recblr
    return recblr


def header_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(recblr_\w+)\(", text, re.M)))


def test_header_declares_the_entry_points():
    syms = header_symbols()
    assert "recblr_bdlru_scan_forward" in syms and "recblr_bdlru_backward" in syms
    assert len(syms) == 23


def test_library_exports_every_declared_symbol(rb):
    import ctypes
    lib = ctypes.CDLL(rb.LIB_PATH)
    for s in header_symbols():
        assert hasattr(lib, s), s
    assert set(header_symbols()) == set(rb.EXPORTS)


def test_status_strings(rb):
    for code in (0, -1, -2, -3, -4, -5):
        assert rb.recblr_status_string(code)
    assert rb.recblr_status_string(99) == b"unknown status"


def test_workspace_sizes(rb):
    assert rb.recblr_workspace_size(rb.OP_SCAN_FORWARD, 256, 2048, 128, rb.F32) == 0
    bwd = rb.recblr_workspace_size(rb.OP_SCAN_BACKWARD, 256, 2048, 128, rb.F32)
    assert bwd >= 256 * 128 * 4
    full = rb.recblr_workspace_size(rb.OP_FORWARD, 4, 50, 64, rb.BF16)
    assert full >= 2 * 4 * 50 * 64 * 2
    assert rb.recblr_workspace_size(rb.OP_STEP, 8, 123, 64, rb.F32) >= 2 * 8 * 64 * 4
    assert rb.recblr_workspace_size(rb.OP_SCAN_FORWARD, -1, 5, 5, rb.F32) == 0
    assert rb.recblr_workspace_size(rb.OP_FORWARD, 1, 5, 5, 9) == 0
    assert rb.recblr_workspace_size(17, 1, 5, 5, rb.F32) == 0


A = 0x10000000  # fake, well aligned device addresses, 64 MiB apart
def addr(k):
    return A + k * (64 << 20)


def scan_fwd(rb, x=addr(0), zr=addr(1), zi=addr(2), lam=addr(3), h0=None, h=addr(4), hT=addr(5),
             B=2, L=3, D=4, io=0, ws=None, nws=0):
    return rb.recblr_bdlru_scan_forward(x, zr, zi, lam, h0, h, hT, B, L, D, io, ws, nws, None)


def test_scan_forward_validation(rb):
    assert scan_fwd(rb, B=-1) == rb.ERR_INVALID_ARGUMENT
    assert scan_fwd(rb, L=-5) == rb.ERR_INVALID_ARGUMENT
    assert scan_fwd(rb, io=2) == rb.ERR_UNSUPPORTED
    assert scan_fwd(rb, x=None) == rb.ERR_INVALID_ARGUMENT
    assert scan_fwd(rb, lam=None) == rb.ERR_INVALID_ARGUMENT
    assert scan_fwd(rb, zr=addr(1) + 2) == rb.ERR_INVALID_ARGUMENT          # misaligned f32
    assert scan_fwd(rb, h=addr(0) + 8) == rb.ERR_INVALID_ARGUMENT            # h overlaps x
    assert scan_fwd(rb, hT=addr(4) + 4) == rb.ERR_INVALID_ARGUMENT           # hT inside h
    assert scan_fwd(rb, B=1 << 31) == rb.ERR_UNSUPPORTED
    # empty problems are accepted without touching anything
    assert scan_fwd(rb, B=0, x=None, zr=None, zi=None, lam=None, h=None) == rb.OK
    assert scan_fwd(rb, D=0, x=None, zr=None, zi=None, lam=None, h=None) == rb.OK


def test_scan_backward_validation(rb):
    def call(**kw):
        a = dict(x=addr(0), zr=addr(1), zi=addr(2), lam=addr(3), h0=None, h=addr(4),
                 dh=addr(5), dhT=None, dx=addr(6), dzr=addr(7), dzi=addr(8), dlam=addr(9),
                 dh0=None, B=2, L=3, D=4, io=0, ws=addr(10), nws=1 << 20)
        a.update(kw)
        return rb.recblr_bdlru_scan_backward(
            a["x"], a["zr"], a["zi"], a["lam"], a["h0"], a["h"], a["dh"], a["dhT"], a["dx"],
            a["dzr"], a["dzi"], a["dlam"], a["dh0"], a["B"], a["L"], a["D"], a["io"], a["ws"],
            a["nws"], None)
    assert call(dlam=None) == rb.ERR_INVALID_ARGUMENT
    assert call(dh=None) == rb.ERR_INVALID_ARGUMENT
    assert call(dzr=addr(6)) == rb.ERR_INVALID_ARGUMENT                     # dzr == dx
    assert call(dx=addr(4)) == rb.ERR_INVALID_ARGUMENT                      # dx over h
    assert call(ws=None) == rb.ERR_WORKSPACE
    assert call(nws=16) == rb.ERR_WORKSPACE
    assert call(ws=addr(10) + 64) == rb.ERR_WORKSPACE                       # not 256-aligned
    assert call(io=5) == rb.ERR_UNSUPPORTED


def test_timed_scan_validation(rb):
    """The measurement variants validate exactly as the plain scans (events untouched)."""
    ev = (addr(20), addr(21))  # never recorded: every call below fails validation
    f = lambda **kw: rb.recblr_bdlru_scan_forward_timed(
        kw.get("x", addr(0)), addr(1), addr(2), kw.get("lam", addr(3)), None, addr(4), None,
        2, kw.get("L", 3), 4, kw.get("io", 0), None, 0, None, *ev)
    assert f(x=None) == rb.ERR_INVALID_ARGUMENT
    assert f(lam=None) == rb.ERR_INVALID_ARGUMENT
    assert f(L=-1) == rb.ERR_INVALID_ARGUMENT
    assert f(io=7) == rb.ERR_UNSUPPORTED
    g = lambda **kw: rb.recblr_bdlru_scan_backward_timed(
        addr(0), addr(1), addr(2), addr(3), None, addr(4), addr(5), None, addr(6),
        kw.get("dzr", addr(7)), addr(8), kw.get("dlam", addr(9)), None, 2, 3, 4, 0,
        kw.get("ws", addr(10)), 1 << 20, None, *ev)
    assert g(dlam=None) == rb.ERR_INVALID_ARGUMENT
    assert g(dzr=addr(6)) == rb.ERR_INVALID_ARGUMENT
    assert g(ws=None) == rb.ERR_WORKSPACE


def test_step_validation(rb):
    def call(h_prev=addr(4), h_next=addr(5), **kw):
        a = dict(x=addr(0), zr=addr(1), zi=addr(2), lam=addr(3), B=8, D=16, io=1)
        a.update(kw)
        return rb.recblr_bdlru_scan_step(a["x"], a["zr"], a["zi"], a["lam"], h_prev, h_next,
                                         a["B"], a["D"], a["io"], None)
    assert call(h_next=addr(4) + 4) == rb.ERR_INVALID_ARGUMENT              # partial overlap
    assert call(h_next=addr(0)) == rb.ERR_INVALID_ARGUMENT                  # over x
    assert call(h_prev=None) == rb.ERR_INVALID_ARGUMENT
    assert call(x=addr(0) + 1) == rb.ERR_INVALID_ARGUMENT                   # misaligned bf16
    assert call(io=3) == rb.ERR_UNSUPPORTED


def test_full_api_validation(rb):
    def fwd(**kw):
        a = dict(x=addr(0), Wr=addr(1), br=None, Wi=addr(2), bi=None, lam=addr(3), h0=None,
                 h=addr(4), hT=None, B=2, L=3, D=4, io=0, ws=addr(6), nws=1 << 20)
        a.update(kw)
        return rb.recblr_bdlru_forward(a["x"], a["Wr"], a["br"], a["Wi"], a["bi"], a["lam"],
                                       a["h0"], a["h"], a["hT"], a["B"], a["L"], a["D"], a["io"],
                                       a["ws"], a["nws"], None)
    assert fwd(D=1025) == rb.ERR_UNSUPPORTED
    assert fwd(Wr=None) == rb.ERR_INVALID_ARGUMENT
    assert fwd(nws=8) == rb.ERR_WORKSPACE
    assert fwd(ws=addr(4)) == rb.ERR_INVALID_ARGUMENT                      # ws over h
    B, D = 3, 8
    need = rb.recblr_workspace_size(rb.OP_STEP, B, 1, D, rb.F32)
    assert rb.recblr_bdlru_step(addr(0), addr(1), None, addr(2), None, addr(3), addr(4), addr(5),
                                B, D, rb.F32, addr(6), need - 1, None) == rb.ERR_WORKSPACE


def test_linear_scan_validation(rb):
    assert rb.recblr_linear_scan_forward(None, addr(1), None, addr(2), None, 2, 3, 4,
                                         None) == rb.ERR_INVALID_ARGUMENT
    assert rb.recblr_linear_scan_forward(addr(0), addr(1), None, addr(1), None, 2, 3, 4,
                                         None) == rb.ERR_INVALID_ARGUMENT


def test_scan_method_validation(rb):
    """Ablation entry: checks run before any launch."""
    f = rb.recblr_scan_forward_method
    assert f(7, addr(0), addr(1), addr(2), addr(3), addr(4), 2, 3, 4, rb.F32, None, 0,
             None) == rb.ERR_INVALID_ARGUMENT                           # unknown method
    assert f(rb.SCAN_TREE, addr(0), addr(1), addr(2), addr(3), addr(4), 2, 5000, 4, rb.F32,
             None, 0, None) == rb.ERR_UNSUPPORTED                       # tree longer than 4096
    assert f(rb.SCAN_SERIAL, None, addr(1), addr(2), addr(3), addr(4), 2, 3, 4, rb.F32, None, 0,
             None) == rb.ERR_INVALID_ARGUMENT                           # null x
    assert f(rb.SCAN_TREE, addr(0), addr(1), addr(2), addr(3), addr(0), 2, 3, 4, rb.F32, None, 0,
             None) == rb.ERR_INVALID_ARGUMENT                           # h over x
    assert f(rb.SCAN_SERIAL, addr(0), addr(1), addr(2), addr(3), addr(4), 2, 3, 4, 5, None, 0,
             None) == rb.ERR_UNSUPPORTED                                # unknown dtype
    assert f(rb.SCAN_TREE, None, None, None, None, None, 0, 3, 4, rb.F32, None, 0,
             None) == rb.OK                                             # empty batch


def test_scan_backward_method_validation(rb):
    """Backward of the ablation's scans: checks run before any launch."""
    f = rb.recblr_scan_backward_method

    def call(method=rb.SCAN_SERIAL, x=addr(0), dx=addr(6), B=2, L=3, D=4, io=rb.F32, nws=1 << 20):
        return f(method, x, addr(1), addr(2), addr(3), addr(4), addr(5), dx, addr(7), addr(8),
                 addr(9), B, L, D, io, addr(10), nws, None)
    assert call(method=7) == rb.ERR_INVALID_ARGUMENT          # unknown method
    assert call(method=rb.SCAN_TREE, L=5000) == rb.ERR_UNSUPPORTED  # tree longer than 4096
    assert call(x=None) == rb.ERR_INVALID_ARGUMENT              # null x
    assert call(dx=addr(0)) == rb.ERR_INVALID_ARGUMENT          # dx over x
    assert call(io=5) == rb.ERR_UNSUPPORTED                     # unknown dtype
    assert call(nws=0) == rb.ERR_WORKSPACE                      # workspace too small
    need = rb.recblr_workspace_size(rb.OP_SCAN_BACKWARD_METHOD, 2, 3, 4, rb.F32)
    assert need >= rb.recblr_workspace_size(rb.OP_SCAN_BACKWARD, 2, 3, 4, rb.F32)


def test_gated_forward_validation(rb):
    def call(K=2, conv_w=addr(7), nws=1 << 20, hx=addr(0)):
        return rb.recblr_gated_forward(hx, addr(1), conv_w, None, K, addr(2), None, addr(3), None,
                                       addr(4), None, addr(5), None, None, 2, 3, 64, rb.F32,
                                       addr(6), nws, None)
    assert call(K=0) == rb.ERR_UNSUPPORTED
    assert call(K=5) == rb.ERR_UNSUPPORTED
    assert call(conv_w=None) == rb.ERR_INVALID_ARGUMENT
    assert call(hx=None) == rb.ERR_INVALID_ARGUMENT
    assert call(nws=16) == rb.ERR_WORKSPACE
    assert rb.recblr_workspace_size(rb.OP_GATED_FORWARD, 2, 3, 64, rb.F32) > 0


def test_gated_backward_validation(rb):
    def call(K=2, conv_w=addr(7), dconv_w=addr(11), nws=1 << 26, hx=addr(0), dhx=addr(12),
             dlam=addr(17), ws=addr(20)):
        return rb.recblr_gated_backward(
            hx, addr(1), conv_w, None, K, addr(2), None, addr(3), None, addr(4), None, addr(5),
            addr(6), None, dhx, addr(13), dconv_w, None, addr(14), addr(15), addr(16),
            addr(18), dlam, None, 2, 3, 64, rb.F32, ws, nws, None)
    assert call(K=0) == rb.ERR_UNSUPPORTED
    assert call(K=5) == rb.ERR_UNSUPPORTED
    assert call(conv_w=None) == rb.ERR_INVALID_ARGUMENT
    assert call(dconv_w=None) == rb.ERR_INVALID_ARGUMENT
    assert call(hx=None) == rb.ERR_INVALID_ARGUMENT
    assert call(dlam=None) == rb.ERR_INVALID_ARGUMENT
    assert call(dhx=addr(0)) == rb.ERR_INVALID_ARGUMENT                    # dhx over hx
    assert call(dconv_w=addr(7)) == rb.ERR_INVALID_ARGUMENT                # over conv_w
    assert call(nws=16) == rb.ERR_WORKSPACE
    assert call(ws=addr(1)) == rb.ERR_INVALID_ARGUMENT                     # ws over hz
    need = rb.recblr_workspace_size(rb.OP_GATED_BACKWARD, 2, 3, 64, rb.F32)
    assert need >= rb.recblr_workspace_size(rb.OP_BACKWARD, 2, 3, 64, rb.F32) + 3 * 2 * 3 * 64 * 4


def test_model_layout_matches_the_oracle(rb):
    """The library's parameter offsets against the oracle's own reading of the
    documented order (two implementations of one layout)."""
    from oracle import model as om
    for D, E, V, layers, K in ((64, 2, 3416, 2, 4), (128, 1, 5, 1, 2), (64, 3, 211, 3, 3)):
        dims = rb.model_dims(2, 3, D, E, V, layers, K)
        lay, total = om.layout(D, E, V, layers, K)
        assert rb.model_param_offsets(dims) == [o for _, _, o in lay]
        assert rb.recblr_model_param_count(dims) == total


def test_model_validation(rb):
    import ctypes
    ok = rb.model_dims(2, 3, 64)
    assert rb.recblr_model_param_count(rb.model_dims(2, 3, 48)) == 0        # D not 64/128/256
    assert rb.recblr_model_param_count(rb.model_dims(2, 3, 64, K=5)) == 0
    assert rb.recblr_model_param_count(rb.model_dims(2, 3, 64, E=17)) == 0   # E*D > 1024
    assert rb.recblr_model_param_offsets(rb.model_dims(0, 3, 64), None, 0) == -1
    def step(m, params=addr(0), ids=addr(1), grads=addr(3), ws=addr(5), nws=1 << 40,
             opts=None):
        o = ctypes.byref(opts) if opts is not None else None
        return rb.recblr_model_train_step(ctypes.byref(m), o, params, ids, addr(2), grads,
                                          addr(4), ws, nws, addr(6), None)
    assert step(rb.model_dims(2, 3, 48)) == rb.ERR_UNSUPPORTED
    assert step(ok, params=None) == rb.ERR_INVALID_ARGUMENT
    assert step(ok, params=addr(0) + 4) == rb.ERR_INVALID_ARGUMENT          # not 256-aligned
    assert step(ok, grads=addr(0)) == rb.ERR_INVALID_ARGUMENT               # grads over params
    # dropout outside [0, 1) (NaN included) and a padding id outside [-1, V)
    for p, pad in ((1.0, -1), (-0.1, -1), (float("nan"), -1), (0.2, -2), (0.2, ok.V)):
        assert step(ok, opts=rb.ModelStepOpts(p, pad, 0, 0)) == rb.ERR_INVALID_ARGUMENT, (p, pad)
    assert rb.recblr_adam_update(addr(0), addr(1), addr(2), addr(3), 10, 0, 1e-3, 0.9, 0.999,
                                 1e-8, None) == rb.ERR_INVALID_ARGUMENT    # step < 1
    assert rb.recblr_adam_update(addr(0), addr(0), addr(2), addr(3), 10, 1, 1e-3, 0.9, 0.999,
                                 1e-8, None) == rb.ERR_INVALID_ARGUMENT    # grads == params



def test_noalloc_rejects_problems_beyond_its_static_scratch(rb):
    """256 x 65536 x 128 fp32 needs ~200 MiB of look-back state and dLambda
    partials, past the 16 MiB static array: rejected before any HIP call."""
    B, L, D = 256, 65536, 128
    assert rb.recblr_workspace_size(rb.OP_SCAN_BACKWARD, B, L, D, rb.F32) > 16 << 20
    big = 1 << 34  # tensors of 8 GiB: fake addresses 16 GiB apart
    a = lambda k: (1 << 40) + k * big
    st = rb.recblr_bdlru_scan_backward_noalloc(a(0), a(1), a(2), a(3), None, a(4), a(5), None,
                                               a(6), a(7), a(8), a(9), None, B, L, D, rb.F32,
                                               None)
    assert st == rb.ERR_SCRATCH
    # invalid arguments are reported first, as by the workspace entry point
    st = rb.recblr_bdlru_scan_backward_noalloc(a(0), a(1), a(2), a(3), None, a(4), a(5), None,
                                               a(0), a(7), a(8), a(9), None, B, L, D, rb.F32,
                                               None)
    assert st == rb.ERR_INVALID_ARGUMENT
