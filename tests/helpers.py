"""Shared helpers of the GPU parity tests: device transfer and the error metric.

Error metric (the tolerance the workloads state, "max relative error", read
with a floor so that it stays meaningful where h crosses zero): per output
tensor, err = max_i |g_i - o_i| / (|o_i| + rms(o)).  Bars: 1e-4 for fp32 I/O,
1e-2 for bf16 I/O with an fp32 state.
"""
import numpy as np

TOL = {"f32": 1e-4, "bf16": 1e-2}


def floored_rel_err(got, want):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if want.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(want * want)))
    denom = np.abs(want) + rms
    if rms == 0.0:
        return float(np.max(np.abs(got - want)))
    return float(np.max(np.abs(got - want) / denom))


def error_report(got, want):
    """Three views of the error of one output tensor: the floored relative
    error the bar applies to, the same with a floor of 1e-3 rms (close to a
    plain elementwise relative error wherever |want| is not tiny), and the
    normwise max|g - o| / max|o|."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if want.size == 0:
        return {"floored": 0.0, "tight": 0.0, "normwise": 0.0}
    diff = np.abs(got - want)
    rms = float(np.sqrt(np.mean(want * want)))
    mx = float(np.max(np.abs(want)))
    return {"floored": float(np.max(diff / (np.abs(want) + rms))) if rms else float(diff.max()),
            "tight": float(np.max(diff / (np.abs(want) + 1e-3 * rms))) if rms else float(diff.max()),
            "normwise": float(diff.max() / mx) if mx else float(diff.max())}


def report(tag, got, want):
    """Print the error report of one output (collected from the GPU logs)."""
    r = error_report(got, want)
    print(f"ERR {tag}: floored {r['floored']:.2e} tight {r['tight']:.2e} "
          f"normwise {r['normwise']:.2e}", flush=True)
    return r


def assert_close(got, want, io, name=""):
    err = floored_rel_err(got, want)
    assert np.all(np.isfinite(np.asarray(got, dtype=np.float64))), f"{name}: non-finite output"
    assert err <= TOL[io], f"{name}: floored relative error {err:.3e} > {TOL[io]:.0e}"
    return err


def dev(a, io="f32"):
    """numpy float32 array (bf16-representable when io == 'bf16') -> GPU tensor of the I/O dtype."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if io == "bf16":
        t = t.to(torch.bfloat16)  # exact: the values are already bf16
    return t.cuda()


def dev32(a):
    import torch
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host(t):
    import torch
    return t.detach().to(torch.float32).cpu().numpy()
