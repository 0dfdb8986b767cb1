"""Benchmark of the BD-LRU scan on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c4]
                    [--api scan|full|step|scan_step|ablation|gated|model]

A step is one pass of the hot path over one batch: the gated scan forward
(recblr_bdlru_scan_forward) followed by its backward
(recblr_bdlru_scan_backward), on synthetic inputs already resident in HBM.
The default workload is the long-history batch B=256, L=2048, D=128 in fp32.
With --api full the step is the whole layer instead: the gate projections and
the scan, forward (recblr_bdlru_forward) and backward (recblr_bdlru_backward,
which recomputes the projections and returns dx, dW, db, dLambda).  With
--api step (default workload c5dec) a step is one recurrent decode step over
the batch with the gate projections fused in (recblr_bdlru_step, state
updated in place); --api scan_step times the same step from precomputed
pre-activations (recblr_bdlru_scan_step).  --api ablation times the layer
forward (gate projections + scan) with the scan algorithms of the paper's
efficiency ablation (serial scan; two-tree scan with sequence padding or with
embedding padding; the production chunked scan) at the paper's three
sequence lengths.  --api gated times the gated recurrent layer core forward
and backward (causal conv + SiLU, BD-LRU with projections, SiLU output gate;
recblr_gated_forward / recblr_gated_backward) on the workload.  --api model
times a full 2-layer RecBLR training step (embedding, behaviour-modelling
layers, softmax cross entropy, backward, Adam) at the MovieLens-1M training
shape of the paper (B=2048, T=200, D=64, E=2, 3,416 items) with its setting
of dropout 0.2 and rows of the dataset's length mix, left-padded; its
roofline is matrix-multiply flops against the fp32 matrix-core peak.
Prints ONE JSON line (metric, value, roofline of the dominant kernel, and the
fp64 CPU oracle timed on a bounded sample of the same workload).  `value` and
`ms_per_step` come from K steps timed back to back with no events in between
(a HIP event costs about 5 us of stream time on each side of what it
brackets).  With the scan API the roofline takes the scan kernel's own
duration, from a HIP event pair that the library stamps with that kernel's
dispatch start and end (recblr_bdlru_scan_*_timed), over K further steps; the
other APIs report it for the whole call, from an event pass of their own.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E peak, GB/s
# Algorithmic HBM bytes per element (B*L*D) of each call, in units of the I/O
# element size.  Scan level -- forward: read x, z_r, z_i; write h.  backward:
# read dh, x, z_r, z_i, h; write dx, dz_r, dz_i.  Full layer (gate projections
# included; the weights are negligible) -- forward: read x; write h.
# backward: read x, h, dh; write dx.
ARRAYS = {"scan": (4, 8), "full": (2, 4)}


# HBM traffic per launch from rocprofv3 counters (FETCH_SIZE scaled by 2.0 and
# WRITE_SIZE by 1.0, the factors a plain 1 GiB device copy reads for them),
# valid only for the kernel sources they were taken on: the sha256 prefix of
# the listed files must match, else the traffic is reported as null.
TRAFFIC = {
    ("c4", "scan_bwd"): {"bytes": 2186777600, "sha": "0208a2897c4c00c7",
                         "sources": ["scan_bwd.hip", "device_common.hpp", "lookback.hpp"]},
    ("c4", "scan_fwd"): {"bytes": 1074241536, "sha": "a62592a42f205fc1",
                         "sources": ["scan_fwd.hip", "device_common.hpp", "lookback.hpp"]},
    ("c5", "scan_bwd"): {"bytes": 1120493568, "sha": "0208a2897c4c00c7",
                         "sources": ["scan_bwd.hip", "device_common.hpp", "lookback.hpp"]},
    ("c5", "scan_fwd"): {"bytes": 582594560, "sha": "a62592a42f205fc1",
                         "sources": ["scan_fwd.hip", "device_common.hpp", "lookback.hpp"]},
}


def traffic_bytes(workload, kernel):
    import hashlib
    rec = TRAFFIC.get((workload, kernel))
    if rec is None:
        return None
    h = hashlib.sha256()
    for f in rec["sources"]:
        with open(os.path.join(ROOT, "paper_2406_12580_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return rec["bytes"] if h.hexdigest()[:16] == rec["sha"] else None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(cfg, api="scan", target_s=10.0):
    """fp64 oracle (forward + backward) on a bounded sample of the workload.

    The sample is the first `rows` batch rows (each row is independent), grown
    until one pass takes a few seconds; whole passes are then repeated until
    about target_s seconds of CPU work have been timed.
    """
    import oracle
    from paper_2406_12580_amd import datagen as dg
    per_row = cfg.L * cfg.D
    if api == "full":
        f = dg.full_inputs(cfg.B, cfg.L, cfg.D, cfg.seed, io=cfg.io, a_range=cfg.a_range,
                           bias=True, grad=True)

        def run(rows):
            s = slice(0, rows)
            t0 = time.perf_counter()
            oracle.forward(f.x[s], f.Wr, f.br, f.Wi, f.bi, f.lam)
            oracle.backward(f.x[s], f.Wr, f.br, f.Wi, f.bi, f.lam, f.dh[s])
            return time.perf_counter() - t0
    else:
        inp = dg.config_inputs(cfg, grad=True)

        def run(rows):
            s = slice(0, rows)
            t0 = time.perf_counter()
            oracle.scan_forward(inp.x[s], inp.zr[s], inp.zi[s], inp.lam)
            oracle.scan_backward(inp.x[s], inp.zr[s], inp.zi[s], inp.lam, inp.dh[s])
            return time.perf_counter() - t0

    rows = 1
    dt = run(rows)
    while dt < target_s / 4 and rows < cfg.B:
        rows = min(cfg.B, max(rows * 2, int(rows * (target_s / 3) / max(dt, 1e-3))))
        dt = run(rows)
    passes, total = 1, dt
    while total < target_s:
        total += run(rows)
        passes += 1
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    out = {"value": passes * rows * per_row / total, "unit": "elements/s", "cores": threads,
           "kind": "oracle",
           "sample": f"fp64 oracle {'layer' if api == 'full' else 'scan'} forward+backward "
                     f"over {rows} of {cfg.B} batch rows "
                     f"(L={cfg.L}, D={cfg.D}), {passes} passes, {total:.1f} s",
           "cpu_model": cpu_model()}
    if api == "scan":
        out["single_thread"] = single_thread_oracle()
    return out


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo, as lscpu reports it)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


_ONE_THREAD = """
import sys, time
sys.path.insert(0, {root!r})
import oracle
from paper_2406_12580_amd import datagen as dg
for name in ("c1", "c2"):
    cfg = dg.CONFIGS[name]
    inp = dg.config_inputs(cfg, grad=True)
    n, t0 = 0, time.perf_counter()
    while True:
        oracle.scan_forward(inp.x, inp.zr, inp.zi, inp.lam)
        oracle.scan_backward(inp.x, inp.zr, inp.zi, inp.lam, inp.dh)
        n += 1
        dt = time.perf_counter() - t0
        if dt > 1.0:
            break
    print(name, n * cfg.B * cfg.L * cfg.D / dt, flush=True)
"""


def single_thread_oracle():
    """fp64 oracle scan forward+backward on one thread (OMP_NUM_THREADS=1, a
    child process) for the two small workloads, in elements/s."""
    import subprocess
    env = dict(os.environ, OMP_NUM_THREADS="1")
    res = subprocess.run([sys.executable, "-c", _ONE_THREAD.format(root=ROOT)], env=env,
                         capture_output=True, text=True, timeout=300)
    out = {}
    for line in res.stdout.splitlines():
        name, v = line.split()
        out[name] = float(v)
    return out


# Shapes of the paper's efficiency ablation: sequence lengths 200, 100 and 257
# (padded to 256, 128 and 512 for the tree scan), training batches 2048, 2048
# and 512, BD-LRU width E * D = 2 * 64; plus a long-history shape.
ABLATION_WORKLOADS = [("ml1m-like", 2048, 200, 128), ("gowalla-like", 2048, 100, 128),
                      ("xlong-like", 512, 257, 128),
                      # few channels, long histories: where parallelism along the
                      # sequence matters (4096 channels, one wave each for the serial scan)
                      ("long-history", 16, 4096, 256)]


def gated_main(args, torch, dg, rb):
    """Gated recurrent layer core (conv taps K = 4) forward + backward on a workload."""
    cfg = dg.CONFIGS[args.workload or "c5"]
    B, L, D = cfg.B, cfg.L, cfg.D
    dev = torch.device("cuda:0")
    dtype = torch.float32 if cfg.io == "f32" else torch.bfloat16
    log(f"generating {cfg.name}: B={B} L={L} D={D} {cfg.io} (gated layer core)")
    f = dg.full_inputs(B, L, D, cfg.seed, io=cfg.io, a_range=cfg.a_range, bias=True, grad=True)
    rng = np.random.default_rng(cfg.seed + 1)
    hz = rng.standard_normal((B, L, D), dtype=np.float32)
    w = (rng.standard_normal((D, 4)) * 0.5).astype(np.float32)
    cb = (rng.standard_normal(D) * 0.1).astype(np.float32)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dtype)
    HX, HZ, Wr, br, Wi, bi, DY = T(f.x), T(hz), T(f.Wr), T(f.br), T(f.Wi), T(f.bi), T(f.dh)
    W4, CB, lam = (torch.from_numpy(a).to(dev) for a in (w, cb, f.lam))
    y, h = torch.empty_like(HX), torch.empty_like(HX)
    dhx, dhz = torch.empty_like(HX), torch.empty_like(HX)
    f32 = dict(dtype=torch.float32, device=dev)
    dW4, dCB, dWr, dWi = (torch.empty(sh, **f32) for sh in ((D, 4), D, (D, D), (D, D)))
    dbr, dbi, dlam = (torch.empty(D, **f32) for _ in range(3))
    io = rb.io_code(dtype)
    nf = rb.recblr_workspace_size(rb.OP_GATED_FORWARD, B, L, D, io)
    nb = rb.recblr_workspace_size(rb.OP_GATED_BACKWARD, B, L, D, io)
    wsf = torch.empty(max(nf, 1), dtype=torch.uint8, device=dev)
    wsb = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)
    s = torch.cuda.current_stream()
    p = lambda t: t.data_ptr()

    def fwd():
        st = rb.recblr_gated_forward(p(HX), p(HZ), p(W4), p(CB), 4, p(Wr), p(br), p(Wi), p(bi),
                                     p(lam), None, p(y), p(h), None, B, L, D, io, p(wsf), nf,
                                     s.cuda_stream)
        assert st == 0, st

    def bwd():
        st = rb.recblr_gated_backward(p(HX), p(HZ), p(W4), p(CB), 4, p(Wr), p(br), p(Wi), p(bi),
                                      p(lam), None, p(h), p(DY), None, p(dhx), p(dhz), p(dW4),
                                      p(dCB), p(dWr), p(dbr), p(dWi), p(dbi), p(dlam), None,
                                      B, L, D, io, p(wsb), nb, s.cuda_stream)
        assert st == 0, st
    for _ in range(args.warmup):
        fwd()
        bwd()
    torch.cuda.synchronize()
    K = args.steps
    t0 = time.perf_counter()
    for k in range(K):
        fwd()
        bwd()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # call split from a separate, untimed pass with events around the calls
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    for k in range(K):
        ev[k][0].record(s)
        fwd()
        ev[k][1].record(s)
        bwd()
        ev[k][2].record(s)
    torch.cuda.synchronize()
    t_f = np.array([ev[k][0].elapsed_time(ev[k][1]) for k in range(K)]) * 1e-3
    t_b = np.array([ev[k][1].elapsed_time(ev[k][2]) for k in range(K)]) * 1e-3
    N = B * L * D
    esz = 4 if cfg.io == "f32" else 2
    # Boundary bytes: forward reads hx, hz and writes y, h; backward reads hx,
    # hz, h, dy and writes dhx, dhz.
    f_gbs = 4 * esz * N / float(np.mean(t_f)) / 1e9
    b_gbs = 6 * esz * N / float(np.mean(t_b)) / 1e9
    dom = "backward" if np.mean(t_b) >= np.mean(t_f) else "forward"
    ach = b_gbs if dom == "backward" else f_gbs
    log(f"gated forward {np.mean(t_f)*1e6:.1f} us ({f_gbs:.0f} GB/s), backward "
        f"{np.mean(t_b)*1e6:.1f} us ({b_gbs:.0f} GB/s)")
    out = {"metric": "gated recurrent layer core elements/sec (B*L*D), forward+backward",
           "value": N * K / wall, "unit": "elements/s", "n_gpus": 1, "steps": K,
           "warmup": args.warmup, "ms_per_step": wall / K * 1e3, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": cfg.io,
           "data": "synthetic (seeded normal hx, hz, dL/dy, conv taps; decay bases per the "
                   "paper's initialisation)",
           "config": {"workload": f"{cfg.name}: gated layer core forward+backward (conv K=4), "
                                  f"{cfg.note}",
                      "B": B, "L": L, "D": D, "io": cfg.io, "elements": N},
           "us_forward": float(np.mean(t_f)) * 1e6, "us_backward": float(np.mean(t_b)) * 1e6,
           "roofline": {"bound": "hbm", "kernel": f"gated_{dom}", "achieved": ach,
                        "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": ach / PEAK_HBM_GBS,
                        "traffic": None}}
    if not args.no_cpu_baseline:
        import oracle
        rows, t0, passes = 1, time.perf_counter(), 0
        while time.perf_counter() - t0 < 10.0:
            oracle.gated_backward(f.x[:rows], hz[:rows], w, cb, f.Wr, f.br, f.Wi, f.bi, f.lam,
                                  f.dh[:rows])
            passes += 1
        total = time.perf_counter() - t0
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        out["cpu_baseline"] = {"value": passes * rows * L * D / total, "unit": "elements/s",
                               "cores": threads, "kind": "oracle",
                               "sample": f"fp64 oracle gated forward+backward (the backward "
                                         f"recomputes the forward) over {rows} of {B} batch "
                                         f"rows (L={L}, D={D}), {passes} passes, {total:.1f} s"}
    print(json.dumps(out), flush=True)


def model_flops(d):
    """Matrix-multiply flops of one training step (forward + backward = 3x forward):
    per token and layer the linear layers Wx, Wz (D -> ED), the BD-LRU gate
    projections (ED -> ED, two), Wo (ED -> D) and the PFFN (D -> 4D -> D); per row
    the prediction h_T E^T."""
    ED = d.E * d.D
    per_token = d.layers * 2 * (2 * d.D * ED + 2 * ED * ED + ED * d.D + 8 * d.D * d.D)
    return 3 * (per_token * d.B * d.T + 2 * d.D * d.V * d.B)


def model_main(args, torch, dg, rb):
    """Full RecBLR model training step (forward, backward, Adam) on the MovieLens-1M
    training shape."""
    d = dg.MODEL_CONFIGS[args.workload or "ml1m"]
    dev = torch.device("cuda:0")
    # the paper's MovieLens-1M setting: dropout 0.2 (its dropout study) and
    # rows of the dataset's length mix, left-padded with id 0
    p_drop, pad, min_len = args.dropout, 0, dg.ml1m_min_len(d.T)
    log(f"model {d}, dropout {p_drop}, lengths U{{{min_len}..{d.T}}} left-padded")
    named = dg.model_params(d, 1)
    ids, targets = dg.model_batch(d, 2, min_len=min_len, pad_id=pad)
    rd = rb.model_dims(d.B, d.T, d.D, d.E, d.V, d.layers, d.K, d.eps)
    offs = rb.model_param_offsets(rd)
    # model_params lists the tensors in the documented parameter order
    assert len(offs) == len(named)
    flat = np.zeros(rb.recblr_model_param_count(rd), dtype=np.float32)
    for (name, arr), o in zip(named.items(), offs):
        flat[o:o + arr.size] = arr.ravel()
    P = torch.from_numpy(flat).to(dev)
    G, M1, M2 = torch.empty_like(P), torch.zeros_like(P), torch.zeros_like(P)
    I, Tg = torch.from_numpy(ids).to(dev), torch.from_numpy(targets).to(dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    step = rb.ModelStep(rd)
    n = [0]

    def one():
        # a new Philox offset per step: new dropout masks every step
        step.train_step(P, I, Tg, G, loss, dropout=p_drop, seed=2406, offset=n[0], pad_id=pad)
        n[0] += 1
        rb.adam_update(P, G, M1, M2, n[0])
    for _ in range(args.warmup):
        one()
    torch.cuda.synchronize()
    first = loss.item()
    K = args.steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    t0 = time.perf_counter()
    ev[0].record()
    for k in range(K):
        one()
    ev[1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dts = np.array([ev[0].elapsed_time(ev[1]) / K]) * 1e-3
    tokens = d.B * d.T
    fl = model_flops(d)
    ach = fl / float(np.mean(dts)) / 1e12
    log(f"model step {np.mean(dts)*1e3:.2f} ms, loss {first:.4f} -> {loss.item():.4f}")
    out = {"metric": "RecBLR model training tokens/sec (B*T per step: forward, backward, Adam)",
           "value": tokens * K / wall, "unit": "tokens/s", "n_gpus": 1, "steps": K,
           "warmup": args.warmup, "ms_per_step": wall / K * 1e3, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic (Zipf item ids, row lengths U{%d..%d} left-padded with id 0, "
                   "seeded random-init weights)" % (min_len, d.T),
           "config": {"workload": f"{args.workload or 'ml1m'}: 2-layer RecBLR, MovieLens-1M "
                                  "training shape", "B": d.B, "T": d.T, "D": d.D, "E": d.E,
                      "V": d.V, "layers": d.layers, "K": d.K, "dropout": p_drop,
                      "real_item_fraction": round(float((ids != pad).mean()), 4)},
           "loss_first_last": [first, loss.item()],
           "roofline": {"bound": "mfma", "kernel": "model_step (matrix-multiply flops)",
                        "achieved": ach, "peak": 157.3, "unit": "TFLOP/s", "frac": ach / 157.3,
                        "traffic": None}}
    step.close()
    if not args.no_cpu_baseline:
        from oracle import model as om
        lay, total = om.layout(d.D, d.E, d.V, d.layers, d.K)
        rows, t0, passes = 2, time.perf_counter(), 0
        f64 = np.zeros(total)
        for name, shape, o in lay:
            f64[o:o + int(np.prod(shape))] = named[name].ravel()
        while time.perf_counter() - t0 < 10.0:
            om.train_step(f64, ids[:rows], targets[:rows], d.D, d.E, d.V, d.layers, d.K, d.eps,
                          dropout=p_drop, seed=2406, offset=passes, pad_id=pad)
            passes += 1
        total = time.perf_counter() - t0
        threads = torch.get_num_threads()
        out["cpu_baseline"] = {"value": passes * rows * d.T / total, "unit": "tokens/s",
                               "cores": threads, "kind": "oracle",
                               "sample": f"fp64 oracle model step over {rows} of {d.B} rows "
                                         f"(T={d.T}), {passes} passes, {total:.1f} s"}
    print(json.dumps(out), flush=True)


def ablation_main(args, torch, dg, rb):
    """Layer forward, and forward + backward (the training step the paper's table
    times), per scan algorithm.

    proj(len) is measured as recblr_bdlru_forward minus the production scan at
    that length (and proj_b(len) as recblr_bdlru_backward minus the production
    scan backward); each scheme's time is the projections at its length plus
    its scans:
      serial:   proj(L)  + serial scan(L)
      tree_sp:  proj(P)  + tree scan of inputs left-padded to P (sequence padding)
      tree_ep:  proj(L)  + tree scan padding to P inside (embedding padding)
      chunked:  proj(L)  + production scan(L)          (P = power of two >= L)
    """
    dev = torch.device("cuda:0")
    s = torch.cuda.current_stream()

    def timed(fn, reps):
        for _ in range(max(args.warmup, 1)):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record(s)
        for k in range(reps):
            fn()
            ev[k + 1].record(s)
        torch.cuda.synchronize()
        return float(np.median([ev[k].elapsed_time(ev[k + 1]) for k in range(reps)])) * 1e3

    rows = []
    for name, B, L, D in ABLATION_WORKLOADS:
        P = 1 << (L - 1).bit_length()
        log(f"{name}: B={B} L={L} (padded {P}) D={D} fp32")
        f = dg.full_inputs(B, L, D, 7000 + L, io="f32", bias=True)
        zr = np.einsum("bld,ed->ble", f.x, f.Wr, optimize=True).astype(np.float32) + f.br
        zi = np.einsum("bld,ed->ble", f.x, f.Wi, optimize=True).astype(np.float32) + f.bi
        T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        padw = ((0, 0), (P - L, 0), (0, 0))
        X, ZR, ZI = T(f.x), T(zr), T(zi)
        XP, ZRP, ZIP = T(np.pad(f.x, padw)), T(np.pad(zr, padw) + 0), T(np.pad(zi, padw) + 0)
        Wr, br, Wi, bi, lam = T(f.Wr), T(f.br), T(f.Wi), T(f.bi), T(f.lam)
        reps = max(args.steps, 5)
        t = {}
        t["layer_L"] = timed(lambda: rb.bdlru_forward(X, Wr, br, Wi, bi, lam), reps)
        t["layer_P"] = timed(lambda: rb.bdlru_forward(XP, Wr, br, Wi, bi, lam), reps)
        t["chunked_L"] = timed(lambda: rb.scan_forward_method(rb.SCAN_CHUNKED, X, ZR, ZI, lam), reps)
        t["chunked_P"] = timed(lambda: rb.scan_forward_method(rb.SCAN_CHUNKED, XP, ZRP, ZIP, lam),
                               reps)
        t["serial"] = timed(lambda: rb.scan_forward_method(rb.SCAN_SERIAL, X, ZR, ZI, lam), reps)
        t["tree_sp"] = timed(lambda: rb.scan_forward_method(rb.SCAN_TREE, XP, ZRP, ZIP, lam), reps)
        t["tree_ep"] = timed(lambda: rb.scan_forward_method(rb.SCAN_TREE, X, ZR, ZI, lam), reps)
        # backward: dL/dh ~ N(0, 1); h from the production forward
        g = np.random.default_rng(7100 + L).standard_normal((B, L, D)).astype(np.float32)
        DH, DHP = T(g), T(np.pad(g, padw))
        H = rb.scan_forward_method(rb.SCAN_CHUNKED, X, ZR, ZI, lam)
        HP = rb.scan_forward_method(rb.SCAN_CHUNKED, XP, ZRP, ZIP, lam)
        HL, _ = rb.bdlru_forward(X, Wr, br, Wi, bi, lam)
        HLP, _ = rb.bdlru_forward(XP, Wr, br, Wi, bi, lam)
        bwd = lambda m, *a: rb.scan_backward_method(m, *a)
        t["layer_b_L"] = timed(lambda: rb.bdlru_backward(X, Wr, br, Wi, bi, lam, HL, DH), reps)
        t["layer_b_P"] = timed(lambda: rb.bdlru_backward(XP, Wr, br, Wi, bi, lam, HLP, DHP), reps)
        t["b_chunked_L"] = timed(lambda: bwd(rb.SCAN_CHUNKED, X, ZR, ZI, lam, H, DH), reps)
        t["b_chunked_P"] = timed(lambda: bwd(rb.SCAN_CHUNKED, XP, ZRP, ZIP, lam, HP, DHP), reps)
        t["b_serial"] = timed(lambda: bwd(rb.SCAN_SERIAL, X, ZR, ZI, lam, H, DH), reps)
        t["b_tree_sp"] = timed(lambda: bwd(rb.SCAN_TREE, XP, ZRP, ZIP, lam, HP, DHP), reps)
        t["b_tree_ep"] = timed(lambda: bwd(rb.SCAN_TREE, X, ZR, ZI, lam, H, DH), reps)
        proj_L, proj_P = t["layer_L"] - t["chunked_L"], t["layer_P"] - t["chunked_P"]
        projb_L, projb_P = t["layer_b_L"] - t["b_chunked_L"], t["layer_b_P"] - t["b_chunked_P"]
        row = {"workload": name, "B": B, "L": L, "padded": P, "D": D,
               "us_scan": {k: round(t[k], 1) for k in ("serial", "tree_sp", "tree_ep", "chunked_L")},
               "us_scan_backward": {k: round(t["b_" + k], 1)
                                    for k in ("serial", "tree_sp", "tree_ep", "chunked_L")},
               "us_projection": {"L": round(proj_L, 1), "padded": round(proj_P, 1)},
               "us_projection_backward": {"L": round(projb_L, 1), "padded": round(projb_P, 1)},
               "us_layer_forward": {"serial": round(proj_L + t["serial"], 1),
                                    "tree_sp": round(proj_P + t["tree_sp"], 1),
                                    "tree_ep": round(proj_L + t["tree_ep"], 1),
                                    "chunked": round(t["layer_L"], 1)},
               "us_layer_train": {
                   "serial": round(proj_L + projb_L + t["serial"] + t["b_serial"], 1),
                   "tree_sp": round(proj_P + projb_P + t["tree_sp"] + t["b_tree_sp"], 1),
                   "tree_ep": round(proj_L + projb_L + t["tree_ep"] + t["b_tree_ep"], 1),
                   "chunked": round(t["layer_L"] + t["layer_b_L"], 1)}}
        log(json.dumps(row))
        rows.append(row)
    first = rows[0]["us_layer_train"]
    out = {"metric": "BD-LRU layer forward + backward, serial-scan time over chunked-scan time "
                     "(efficiency-ablation analogue, ml1m-like)",
           "value": first["serial"] / first["chunked"], "unit": "x", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic (seeded normal x, weights N(0, 1/D), decay bases per the paper's "
                   "initialisation)",
           "config": {"workload": "efficiency ablation analogue: ml1m-like, gowalla-like, "
                                  "xlong-like shapes"},
           "table": rows}
    print(json.dumps(out), flush=True)


def decode_main(args, torch, dg, rb):
    """One recurrent step over a decode batch per timed step (state updated in place)."""
    cfg = dg.CONFIGS[args.workload or "c5dec"]
    B, D = cfg.B, cfg.D
    dev = torch.device("cuda:0")
    dtype = torch.float32 if cfg.io == "f32" else torch.bfloat16
    io = rb.io_code(dtype)
    esz = 4 if cfg.io == "f32" else 2
    fused = args.api == "step"
    log(f"generating {cfg.name}: B={B} D={D} {cfg.io} ({args.api})")
    f = dg.full_inputs(B, 1, D, cfg.seed, io=cfg.io, a_range=cfg.a_range, bias=True, h0=True)
    s = torch.cuda.current_stream().cuda_stream
    p = lambda t: t.data_ptr()
    arrays_bytes = (esz + 8) if fused else (3 * esz + 8)  # x (, z_r, z_i); h read and written
    # One step's arrays fit the 256 MB last-level cache (MALL) at this size, so
    # consecutive steps rotate over enough copies (> 600 MB in all) that every
    # step streams its data from HBM.
    nsets = max(1, -(-600_000_000 // (arrays_bytes * B * D)))
    if fused:
        x0 = torch.from_numpy(np.ascontiguousarray(f.x[:, 0])).to(dev).to(dtype)
        lam = torch.from_numpy(f.lam).to(dev)
        h0 = torch.from_numpy(f.h0).to(dev)
        Wr, br, Wi, bi = (torch.from_numpy(a).to(dev).to(dtype) for a in (f.Wr, f.br, f.Wi, f.bi))
        nws = rb.recblr_workspace_size(rb.OP_STEP, B, 1, D, io)
        ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
        sets = [(x0.clone(), h0.clone()) for _ in range(nsets)]

        def step(j):
            x, h = sets[j % nsets]
            st = rb.recblr_bdlru_step(p(x), p(Wr), p(br), p(Wi), p(bi), p(lam), p(h), p(h), B, D,
                                      io, p(ws), nws, s)
            assert st == 0, st
    else:
        si = dg.step_inputs(B, D, cfg.seed, io=cfg.io, a_range=cfg.a_range)
        x0, zr0, zi0 = (torch.from_numpy(a).to(dev).to(dtype) for a in (si.x, si.zr, si.zi))
        lam = torch.from_numpy(si.lam).to(dev)
        h0 = torch.from_numpy(si.h0).to(dev)
        sets = [(x0.clone(), zr0.clone(), zi0.clone(), h0.clone()) for _ in range(nsets)]

        def step(j):
            x, zr, zi, h = sets[j % nsets]
            st = rb.recblr_bdlru_scan_step(p(x), p(zr), p(zi), p(lam), p(h), p(h), B, D, io, s)
            assert st == 0, st
    log(f"{nsets} buffer sets of {arrays_bytes * B * D / 1e6:.0f} MB rotate between steps")
    for j in range(args.warmup):
        step(j)
    torch.cuda.synchronize()
    K = args.steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    stream = torch.cuda.current_stream()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for k in range(K):
        step(args.warmup + k)
    ev[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dts = np.array([ev[0].elapsed_time(ev[1]) / K]) * 1e-3
    N = B * D
    ach = arrays_bytes * N / float(np.mean(dts)) / 1e9
    log(f"step {np.mean(dts)*1e6:.1f} us ({ach:.0f} GB/s)  wall/step {wall/K*1e6:.1f} us")
    out = {
        "metric": "BD-LRU decode elements/sec (B*D per step)"
                  + (", gate projections fused" if fused else ", pre-activations given"),
        "value": N * K / wall, "unit": "elements/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": wall / K * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.io,
        "data": "synthetic (seeded normal x, state; decay bases per the paper's initialisation)",
        "config": {"workload": f"{cfg.name}: one recurrent step, {cfg.note}", "B": B, "D": D,
                   "io": cfg.io, "elements": N},
        "us_step": float(np.mean(dts)) * 1e6,
        "roofline": {"bound": "hbm", "kernel": "step_fused" if fused else "scan_step",
                     "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": ach / PEAK_HBM_GBS, "traffic": None},
    }
    if not args.no_cpu_baseline:
        import oracle
        rows = min(B, 4096)
        t0 = time.perf_counter()
        passes = 0
        if fused:
            xs, hs = f.x[:rows, 0], f.h0[:rows].astype(np.float64)
        else:
            xs, hs = si.x[:rows], si.h0[:rows].astype(np.float64)
        while time.perf_counter() - t0 < 10.0:
            if fused:
                hs = oracle.step(xs, f.Wr, f.br, f.Wi, f.bi, f.lam, hs)
            else:
                hs = oracle.scan_step(xs, si.zr[:rows], si.zi[:rows], si.lam, hs)
            passes += 1
        total = time.perf_counter() - t0
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        out["cpu_baseline"] = {"value": passes * rows * D / total, "unit": "elements/s",
                               "cores": threads, "kind": "oracle",
                               "sample": f"fp64 oracle step over {rows} of {B} batch rows "
                                         f"(D={D}), {passes} steps, {total:.1f} s"}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--api", choices=["scan", "full", "step", "scan_step", "ablation", "gated",
                                      "model"], default="scan")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--dropout", type=float, default=0.2,
                    help="--api model: drop probability (the paper's MovieLens-1M rate)")
    ap.add_argument("--copy-reference", type=int, default=0, metavar="MIB",
                    help="only run K plain device copies of MIB MiB (calibrates HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the BD-LRU path is "
              "built and measured on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2406_12580_amd import datagen as dg
    from paper_2406_12580_amd import recblr as rb

    if args.copy_reference:
        n = args.copy_reference * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(args.warmup + args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_reference_bytes_each_way": 4 * n, "copies": args.warmup + args.steps}))
        return

    if args.api in ("step", "scan_step"):
        return decode_main(args, torch, dg, rb)
    if args.api == "ablation":
        return ablation_main(args, torch, dg, rb)
    if args.api == "gated":
        return gated_main(args, torch, dg, rb)
    if args.api == "model":
        return model_main(args, torch, dg, rb)
    cfg = dg.CONFIGS[args.workload or "c4"]
    if "bwd" not in cfg.ops:
        sys.exit(f"workload {cfg.name} has no backward; pick one of c3, c4, c5")
    dev = torch.device("cuda:0")
    dtype = torch.float32 if cfg.io == "f32" else torch.bfloat16
    log(f"generating {cfg.name}: B={cfg.B} L={cfg.L} D={cfg.D} {cfg.io} ({args.api} API)")
    B, L, D = cfg.B, cfg.L, cfg.D
    N = B * L * D
    io = rb.io_code(dtype)
    esz = 4 if cfg.io == "f32" else 2
    stream = torch.cuda.current_stream()
    s = stream.cuda_stream
    p = lambda t: t.data_ptr()
    hT = torch.empty((B, D), dtype=torch.float32, device=dev)
    dlam = torch.empty(D, dtype=torch.float32, device=dev)
    dh0 = torch.empty((B, D), dtype=torch.float32, device=dev)
    if args.api == "scan":
        inp = dg.config_inputs(cfg, grad=True)
        X, ZR, ZI, DH = (torch.from_numpy(a).to(dev).to(dtype)
                         for a in (inp.x, inp.zr, inp.zi, inp.dh))
        lam = torch.from_numpy(inp.lam).to(dev)
        del inp
        h = torch.empty_like(X)
        dx, dzr, dzi = torch.empty_like(X), torch.empty_like(X), torch.empty_like(X)
        nf = rb.recblr_workspace_size(rb.OP_SCAN_FORWARD, B, L, D, io)
        nb = rb.recblr_workspace_size(rb.OP_SCAN_BACKWARD, B, L, D, io)
        wsf = torch.empty(max(nf, 1), dtype=torch.uint8, device=dev)
        wsb = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)

        # The measurement entry points also record a HIP event pair on the launch
        # stream right around the scan kernel itself (kev[0] forward, kev[1]
        # backward); the pairs of the timed steps give the kernel durations.
        kev = [None, None]

        def fwd():
            e = kev[0] or (None, None)
            st = rb.recblr_bdlru_scan_forward_timed(p(X), p(ZR), p(ZI), p(lam), None, p(h), p(hT),
                                                    B, L, D, io, p(wsf), nf, s, e[0], e[1])
            assert st == 0, st

        def bwd():
            e = kev[1] or (None, None)
            st = rb.recblr_bdlru_scan_backward_timed(p(X), p(ZR), p(ZI), p(lam), None, p(h), p(DH),
                                                     None, p(dx), p(dzr), p(dzi), p(dlam), p(dh0),
                                                     B, L, D, io, p(wsb), nb, s, e[0], e[1])
            assert st == 0, st
    else:
        f = dg.full_inputs(B, L, D, cfg.seed, io=cfg.io, a_range=cfg.a_range, bias=True,
                           grad=True)
        X, Wr, br, Wi, bi, DH = (torch.from_numpy(a).to(dev).to(dtype)
                                 for a in (f.x, f.Wr, f.br, f.Wi, f.bi, f.dh))
        lam = torch.from_numpy(f.lam).to(dev)
        del f
        h, dx = torch.empty_like(X), torch.empty_like(X)
        dWr, dWi = (torch.empty((D, D), dtype=torch.float32, device=dev) for _ in range(2))
        dbr, dbi = (torch.empty(D, dtype=torch.float32, device=dev) for _ in range(2))
        nf = rb.recblr_workspace_size(rb.OP_FORWARD, B, L, D, io)
        nb = rb.recblr_workspace_size(rb.OP_BACKWARD, B, L, D, io)
        wsf = torch.empty(max(nf, 1), dtype=torch.uint8, device=dev)
        wsb = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)

        def fwd():
            st = rb.recblr_bdlru_forward(p(X), p(Wr), p(br), p(Wi), p(bi), p(lam), None, p(h),
                                         p(hT), B, L, D, io, p(wsf), nf, s)
            assert st == 0, st

        def bwd():
            st = rb.recblr_bdlru_backward(p(X), p(Wr), p(br), p(Wi), p(bi), p(lam), None, p(h),
                                          p(DH), None, p(dx), p(dWr), p(dbr), p(dWi), p(dbi),
                                          p(dlam), p(dh0), B, L, D, io, p(wsb), nb, s)
            assert st == 0, st

    for _ in range(args.warmup):
        fwd()
        bwd()
    torch.cuda.synchronize()
    K = args.steps
    kernel_ev = None
    if args.api == "scan":
        # torch creates an event on its first record; record each once so that
        # the raw handles exist before the library uses them.
        kernel_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
        for row in kernel_ev:
            for e in row:
                e.record(stream)
    torch.cuda.synchronize()
    # Timed region: K steps back to back, no events (an event costs about 5 us
    # of stream time on each side of the kernel it brackets).
    t0 = time.perf_counter()
    for k in range(K):
        fwd()
        bwd()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if kernel_ev is not None:
        # Kernel durations: K more steps in which the library stamps kernel_ev
        # with the two scan kernels' own start and end times (taken from their
        # dispatches by hipExtLaunchKernelGGL).
        for k in range(K):
            r = kernel_ev[k]
            kev[0] = (r[0].cuda_event, r[1].cuda_event)
            kev[1] = (r[2].cuda_event, r[3].cuda_event)
            fwd()
            bwd()
        torch.cuda.synchronize()
        kev[0] = kev[1] = None
    # Call split, from a separate pass with an event around each call (each
    # event record costs some stream time, so these passes are not timed).
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    for k in range(K):
        ev[k][0].record(stream)
        fwd()
        ev[k][1].record(stream)
        bwd()
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    t_fwd = np.array([ev[k][0].elapsed_time(ev[k][1]) for k in range(K)]) * 1e-3
    t_bwd = np.array([ev[k][1].elapsed_time(ev[k][2]) for k in range(K)]) * 1e-3
    step_s = wall / K
    fb_s = float(np.mean(t_fwd + t_bwd))
    fwd_arrays, bwd_arrays = ARRAYS[args.api]
    fwd_bytes = fwd_arrays * esz * N
    bwd_bytes = bwd_arrays * esz * N
    fwd_gbs = fwd_bytes / float(np.mean(t_fwd)) / 1e9
    bwd_gbs = bwd_bytes / float(np.mean(t_bwd)) / 1e9
    dom = "bwd" if np.mean(t_bwd) >= np.mean(t_fwd) else "fwd"
    ach = bwd_gbs if dom == "bwd" else fwd_gbs
    kernel_us = None
    if kernel_ev is not None:
        # Roofline of the dominant kernel on its own duration (the call times
        # above include the look-back reset and the dLambda reduction, and the
        # event packets of their pass).
        k_fwd = np.array([r[0].elapsed_time(r[1]) for r in kernel_ev]) * 1e-3
        k_bwd = np.array([r[2].elapsed_time(r[3]) for r in kernel_ev]) * 1e-3
        kernel_us = {"fwd": float(np.mean(k_fwd)) * 1e6, "bwd": float(np.mean(k_bwd)) * 1e6}
        dom = "bwd" if kernel_us["bwd"] >= kernel_us["fwd"] else "fwd"
        ach = (bwd_bytes if dom == "bwd" else fwd_bytes) / (kernel_us[dom] * 1e-6) / 1e9
    log(f"fwd {np.mean(t_fwd)*1e6:.1f} us ({fwd_gbs:.0f} GB/s)  bwd {np.mean(t_bwd)*1e6:.1f} us "
        f"({bwd_gbs:.0f} GB/s)  wall/step {step_s*1e6:.1f} us")

    full = args.api == "full"
    kname = ("layer_" if full else "scan_") + dom
    out = {
        "metric": ("BD-LRU layer (gate projections + scan)" if full else "BD-LRU scan")
                  + " elements/sec (B*L*D), forward+backward",
        "value": N / step_s,
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.io,
        "data": "synthetic (seeded normal x, z, dL/dh; decay bases per the paper's initialisation)",
        "config": {"workload": f"{cfg.name}: BD-LRU {'layer' if full else 'scan'} "
                               f"forward+backward, {cfg.note}",
                   "B": B, "L": L, "D": D, "io": cfg.io, "elements": N},
        "fwd_elements_per_s": N / float(np.mean(t_fwd)),
        "fwd_bwd_elements_per_s_call_events": N / fb_s,
        "us_fwd": float(np.mean(t_fwd)) * 1e6,
        "us_bwd": float(np.mean(t_bwd)) * 1e6,
        "fwd_hbm_gbs": fwd_gbs,
        "bwd_hbm_gbs": bwd_gbs,
        "kernel_us": kernel_us,
        "roofline": {"bound": "hbm", "kernel": kname,
                     "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": ach / PEAK_HBM_GBS,
                     "traffic": traffic_bytes(cfg.name, kname)},
    }
    if not args.no_cpu_baseline:
        log("timing the fp64 CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(cfg, args.api)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
