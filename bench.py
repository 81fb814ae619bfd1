#!/usr/bin/env python3
"""Throughput benchmark of libhexconv on one MI355X.

Default workload (the headline metric's configuration): camera-shaped hex
convolution, fp32, N=256 images of 40x40 (hexagonal 1027-pixel footprint,
log-normal x Bernoulli(0.1) amplitudes), 1 -> 16 channels, kernel size 2
(19 taps), stride 1.  One step = forward, then both gradients (data, and
weight with bias) through the combined backward entry point, over one batch.
Value = effective GFLOP/s counting 2*N*H_out*W_out*C_in*C_out*T for each of
the three products (hex taps only).

Inputs are resident in HBM before timing starts.  The K timed steps are
captured once into a HIP graph and replayed (after W eager warm-up steps and
one untimed replay), so the time is GPU execution, not Python launch cost.  Each step works on a
different batch from a rotating set whose total size exceeds the 256 MB
Infinity Cache, so reads and writes go to HBM rather than staying cached.

Other workloads print their own line on request: --config c1 (the tiny
fp32 forward, N=4, 1 -> 4 channels, 16x16, k=1: launch-latency bound,
reported in microseconds per call as us_per_step), c3 (hex max and
average pooling, bf16, GB/s), c4 (wide-channel bf16 convolution, GFLOP/s)
and c5 (the five-layer bf16 stack, forward and backward, samples/s).

Prints one JSON line.  With --gpus > 1 it exits: the library runs on one GPU.
"""
from __future__ import annotations

import argparse
import hashlib
import glob
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_1903_01814_amd import hexconv as hx          # noqa: E402
from paper_1903_01814_amd import inputs as gen         # noqa: E402

HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
CACHE_BYTES = 256 << 20
ROTATE_MIN_BYTES = 3 * CACHE_BYTES


def source_hash():
    h = hashlib.sha1()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_1903_01814_amd", "csrc", "*"))):
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:12]


def read_counters(workload, kernel):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, if it
    was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "counters_%s.txt" % workload)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            a, b = line.split(":", 1)
            kv[a.strip()] = b.strip()
    if kv.get("source_hash") != source_hash() or kv.get("kernel") != kernel:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


class EagerTimer:
    """Plain launches bracketed by HIP events (used for counter collection,
    where graph replay is not wanted)."""

    def __init__(self, torch):
        self.torch = torch

    def time(self, fn, reps):
        t = self.torch
        t.cuda.synchronize()
        a = t.cuda.Event(enable_timing=True)
        b = t.cuda.Event(enable_timing=True)
        st = t.cuda.current_stream()
        a.record(st)
        for i in range(reps):
            fn(i)
        b.record(st)
        t.cuda.synchronize()
        return a.elapsed_time(b) / reps


class GraphTimer:
    """Captures `reps` calls of a launch sequence into one HIP graph (the
    library enqueues on torch's current stream, which is the capture stream
    inside the capture) and times one replay with HIP events recorded on the
    replay stream.  Host-side launch cost is thereby outside the timed
    region; what remains is GPU execution of the kernels back to back."""

    def __init__(self, torch):
        self.torch = torch

    def time(self, fn, reps):
        t = self.torch
        g = t.cuda.CUDAGraph()
        t.cuda.synchronize()
        with t.cuda.graph(g):
            for i in range(reps):
                fn(i)
        g.replay()                                # upload + untimed first replay
        t.cuda.synchronize()
        a = t.cuda.Event(enable_timing=True)
        b = t.cuda.Event(enable_timing=True)
        st = t.cuda.current_stream()
        a.record(st)
        g.replay()
        b.record(st)
        t.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        del g
        return ms                                 # ms per call


def dominant_kernel(torch, fn, reps):
    """The kernel with the largest GPU time over `reps` eager calls of fn,
    timed by the library (a HIP event pair around every launch, on the
    stream it is launched on).  Returns (name, ms per launch, launches per
    call, {name: ms per launch})."""
    torch.cuda.synchronize()
    hx.hexconv_timing_begin()
    for i in range(reps):
        fn(i)
    t = hx.hexconv_timing_end()
    if not t:
        raise RuntimeError("bench.py: no kernel launch was recorded")
    name = max(t, key=lambda n: t[n][1])
    cnt, tot = t[name]
    return name, tot / cnt, cnt / reps, {n: round(ms / c, 5) for n, (c, ms) in t.items()}


# backward kernels computing both gradients in one pass; every other
# backward kernel computes one of them
BOTH_GRADIENT_KERNELS = ("bwd_smallc_k",)


def products_of(kernel, op):
    """Convolution products (of the three per layer) one launch of `kernel`
    performs when it runs for `op`."""
    if op.endswith("fwd"):
        return 1
    return 2 if kernel in BOTH_GRADIENT_KERNELS else 1


def conv_flop(N, Ci, Co, Ho, Wo, T):
    return 2.0 * N * Ho * Wo * Ci * Co * T


def dev(torch, a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype).to("cuda:0")


def cpu_baseline_conv(cfg, d, k, s, seconds):
    """The fp64 oracle on the same full-batch workload (fwd + bwd), repeated
    until `seconds` of CPU time have elapsed; returns GFLOP/s and threads."""
    import oracle
    H, W = cfg["H"], cfg["W"]
    Ho, Wo = oracle.out_shape(H, W, s)
    T = oracle.num_taps(k)
    has_bwd = "dy" in d
    flop = (3 if has_bwd else 1) * conv_flop(cfg["N"], cfg["C_in"], cfg["C_out"], Ho, Wo, T)
    reps = 0
    t0 = time.perf_counter()
    while True:
        oracle.conv_fwd(d["x"], d["w"], d["b"], k, s)
        if has_bwd:
            oracle.conv_bwd_data(d["dy"], d["w"], k, s, H, W)
            oracle.conv_bwd_weight(d["x"], d["dy"], k, s)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return flop * reps / el / 1e9, oracle.threads(), reps, el


def bench_conv(args, torch, cfg_key):
    cfg = gen.CONFIGS[cfg_key]
    N, Ci, Co, H, W, k, s = (cfg[n] for n in ("N", "C_in", "C_out", "H", "W", "k", "stride"))
    T = hx.hex_num_taps(k)
    Ho, Wo = hx.hex_out_shape(H, W, k, s)
    dt = torch.float32 if cfg["dtype"] == gen.F32 else torch.bfloat16
    esz = 4 if dt == torch.float32 else 2
    per_set = esz * (N * Ci * H * W * 2 + N * Co * Ho * Wo * 2)
    # enough batches to exceed the Infinity Cache (a tiny launch-bound
    # workload stops at 256)
    nsets = min(256, max(1, -(-ROTATE_MIN_BYTES // per_set)))
    d0 = gen.conv_inputs(cfg, T, (Ho, Wo), seed=0)
    sets = []
    for b in range(nsets):
        d = d0 if b == 0 else gen.conv_inputs(cfg, T, (Ho, Wo), seed=b)
        sets.append(dict(x=dev(torch, d["x"], dt),
                         dy=dev(torch, d["dy"], dt) if "dy" in d else None,
                         y=torch.empty((N, Co, Ho, Wo), dtype=dt, device="cuda:0"),
                         dx=torch.empty((N, Ci, H, W), dtype=dt, device="cuda:0")))
        if b == 0:
            w = dev(torch, d["w"], dt)
            bias = dev(torch, d["b"], dt)
    dw = torch.empty((Co, Ci, T), dtype=torch.float32, device="cuda:0")
    db = torch.empty((Co,), dtype=torch.float32, device="cuda:0")
    dtc = hx.HEX_F32 if esz == 4 else hx.HEX_BF16
    nws = max(hx.hexconv_bwd_weight_workspace(N, Ci, Co, H, W, k, s, dtc),
              hx.hexconv_bwd_workspace(N, Ci, Co, H, W, k, s, dtc))
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda:0")
    # the binding enqueues on torch's current stream (the capture stream
    # while a graph is being captured)
    def fwd(i):
        z = sets[i % nsets]
        hx.hexconv_fwd(z["x"], w, bias, z["y"], k, s)

    def bwd(i):
        z = sets[i % nsets]
        hx.hexconv_bwd(z["x"], z["dy"], w, z["dx"], dw, db, ws, k, s)

    def bwd_data(i):
        z = sets[i % nsets]
        hx.hexconv_bwd_data(z["dy"], w, z["dx"], k, s)

    def bwd_weight(i):
        z = sets[i % nsets]
        hx.hexconv_bwd_weight(z["x"], z["dy"], dw, db, ws, k, s)

    has_bwd = bool(cfg.get("bwd"))

    def step(i):
        fwd(i)
        if has_bwd:
            bwd(i)

    timer = EagerTimer(torch) if args.eager else GraphTimer(torch)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_step = timer.time(step, args.steps)

    # per-op durations, each op alone over the same rotation (HIP events on
    # the launch stream); the step uses fwd and bwd, the separate gradient
    # entry points are timed for reference (forward-only workloads: fwd)
    ops = {}
    x_b, y_b = esz * N * Ci * H * W, esz * N * Co * Ho * Wo
    w_b, b_b, g_b = esz * Co * Ci * T, esz * Co, 4 * (Co * Ci * T + Co)
    bytes_alg = {
        "fwd": x_b + w_b + b_b + y_b,
        "bwd": x_b + y_b + w_b + x_b + g_b,          # x, dy, w -> dx, dw, db
        "bwd_data": y_b + w_b + x_b,
        "bwd_weight": x_b + y_b + g_b,
    }
    nprod = {"fwd": 1, "bwd": 2, "bwd_data": 1, "bwd_weight": 1}
    op_list = (("fwd", fwd), ("bwd", bwd), ("bwd_data", bwd_data),
               ("bwd_weight", bwd_weight)) if has_bwd else (("fwd", fwd),)
    for name, fn in op_list:
        ms = timer.time(fn, args.steps)
        ops[name] = dict(ms=ms, gbs=bytes_alg[name] / (ms * 1e-3) / 1e9)
    flop_op = conv_flop(N, Ci, Co, Ho, Wo, T)
    flop_step = (3 if has_bwd else 1) * flop_op
    value = flop_step / (ms_step * 1e-3) / 1e9

    # the dominant op of the step, and within it the kernel with the most
    # GPU time, against its roofline: the op's algorithmic bytes (or
    # products) per launch of that kernel over its measured duration
    dom = max(("fwd", "bwd") if has_bwd else ("fwd",), key=lambda n: ops[n]["ms"])
    fn_dom = fwd if dom == "fwd" else bwd
    kname, kms, kper, kall = dominant_kernel(torch, fn_dom, args.steps)
    bound = "hbm" if cfg["dtype"] == gen.F32 or Ci * T < 64 else "mfma"
    if bound == "hbm":
        units = bytes_alg[dom] / kper
        achieved = units / (kms * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(achieved / HBM_PEAK_GBS, 4))
    else:
        units = products_of(kname, dom) * flop_op / kper
        achieved = units / (kms * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=round(achieved, 2), peak=BF16_MFMA_PEAK_TFLOPS,
                    unit="TFLOP/s", frac=round(achieved / BF16_MFMA_PEAK_TFLOPS, 4))
    roof["traffic"] = read_counters(cfg["name"], kname)
    roof.update(kernel=kname, kernel_ms=round(kms, 5), launches_per_op=kper, op=dom,
                alg_per_launch=units, op_kernels_ms=kall)

    out = dict(
        metric="hex-conv effective GFLOP/s (%s)" % ("fwd+bwd" if has_bwd else "fwd"),
        value=round(value, 2), unit="GFLOP/s",
        n_gpus=1, steps=args.steps, warmup=args.warmup, ms_per_step=round(ms_step, 5),
        higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="f32" if esz == 4 else "bf16", data="synthetic",
        config=dict(workload=cfg["name"], N=N, C_in=Ci, C_out=Co, H=H, W=W, k=k, stride=s,
                    taps=T, H_out=Ho, W_out=Wo, rotating_batches=nsets),
        samples_per_s=round(N / (ms_step * 1e-3), 1),
        us_per_step=round(ms_step * 1e3, 3),
        per_op={n: dict(ms=round(v["ms"], 5), alg_GBps=round(v["gbs"], 1),
                        GFLOPs=round(nprod[n] * flop_op / (v["ms"] * 1e-3) / 1e9, 1))
                for n, v in ops.items()},
        roofline=roof,
    )
    if not args.no_cpu_baseline:
        d = d0
        gfs, thr, reps, el = cpu_baseline_conv(cfg, d, k, s, args.cpu_seconds)
        out["cpu_baseline"] = dict(
            value=round(gfs, 3), unit="GFLOP/s", cores=thr, kind="oracle",
            sample="full batch (N=%d) %s, fp64, repeated %d times in %.1f s"
                   % (N, "fwd+bwd_data+bwd_weight" if has_bwd else "fwd", reps, el))
    return out


def cpu_baseline_pool(cfg, x, seconds):
    """The fp64 oracle's max and average pooling on an 8-image slice,
    repeated for `seconds`; returns GB/s of the same algorithmic bytes."""
    import oracle
    xs = x[:8]
    k, s = cfg["k"], cfg["stride"]
    Ho, Wo = oracle.out_shape(cfg["H"], cfg["W"], s)
    nbytes = 2 * 2 * (xs.size + xs.shape[0] * xs.shape[1] * Ho * Wo)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.pool_fwd(xs, k, s, oracle.POOL_MAX)
        oracle.pool_fwd(xs, k, s, oracle.POOL_AVG)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return nbytes * reps / el / 1e9, oracle.threads(), reps, el


def bench_pool(args, torch, cfg_key):
    cfg = gen.CONFIGS[cfg_key]
    N, C, H, W, k, s = (cfg[n] for n in ("N", "C", "H", "W", "k", "stride"))
    Ho, Wo = hx.hex_out_shape(H, W, k, s)
    dt = torch.bfloat16
    esz = 2
    in_b, out_b = esz * N * C * H * W, esz * N * C * Ho * Wo
    nsets = max(1, -(-ROTATE_MIN_BYTES // (in_b + 2 * out_b)))
    d0 = gen.pool_inputs(cfg, seed=0)
    sets = []
    for b in range(nsets):
        d = d0 if b == 0 else gen.pool_inputs(cfg, seed=b)
        sets.append(dict(x=dev(torch, d["x"], dt),
                         ymax=torch.empty((N, C, Ho, Wo), dtype=dt, device="cuda:0"),
                         yavg=torch.empty((N, C, Ho, Wo), dtype=dt, device="cuda:0")))

    def pmax(i):
        z = sets[i % nsets]
        hx.hexpool_fwd(z["x"], z["ymax"], None, k, s, hx.HEX_POOL_MAX)

    def pavg(i):
        z = sets[i % nsets]
        hx.hexpool_fwd(z["x"], z["yavg"], None, k, s, hx.HEX_POOL_AVG)

    def step(i):
        pmax(i)
        pavg(i)

    timer = EagerTimer(torch) if args.eager else GraphTimer(torch)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_step = timer.time(step, args.steps)
    ops = {}
    for name, fn in (("max", pmax), ("avg", pavg)):
        ms = timer.time(fn, args.steps)
        ops[name] = dict(ms=ms, gbs=(in_b + out_b) / (ms * 1e-3) / 1e9)
    value = 2 * (in_b + out_b) / (ms_step * 1e-3) / 1e9
    dom = max(ops, key=lambda n: ops[n]["ms"])
    kname, kms, kper, kall = dominant_kernel(torch, pmax if dom == "max" else pavg, args.steps)
    units = (in_b + out_b) / kper
    achieved = units / (kms * 1e-3) / 1e9
    roof = dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                frac=round(achieved / HBM_PEAK_GBS, 4))
    roof["traffic"] = read_counters(cfg["name"], kname)
    roof.update(kernel=kname, kernel_ms=round(kms, 5), launches_per_op=kper, op=dom,
                alg_per_launch=units, op_kernels_ms=kall)
    out = dict(
        metric="hex-pool HBM GB/s (max + avg, fwd)", value=round(value, 1), unit="GB/s",
        n_gpus=1, steps=args.steps, warmup=args.warmup, ms_per_step=round(ms_step, 5),
        higher_is_better=True, scaling="weak", vs_baseline=None, dtype="bf16",
        data="synthetic",
        config=dict(workload=cfg["name"], N=N, C=C, H=H, W=W, k=k, stride=s, H_out=Ho,
                    W_out=Wo, rotating_batches=nsets),
        per_op={n: dict(ms=round(v["ms"], 5), alg_GBps=round(v["gbs"], 1))
                for n, v in ops.items()},
        roofline=roof,
    )
    if not args.no_cpu_baseline:
        gbs, thr, reps, el = cpu_baseline_pool(cfg, d0["x"], args.cpu_seconds)
        out["cpu_baseline"] = dict(
            value=round(gbs, 3), unit="GB/s", cores=thr, kind="oracle",
            sample="8 of %d images, max and avg pooling, fp64, repeated %d times in %.1f s"
                   % (N, reps, el))
    return out


def stack_shapes(cfg):
    """Per layer: (kind, C_in, C_out, k, stride, relu, H_in, W_in, H_out, W_out)."""
    H, W = cfg["H"], cfg["W"]
    out = []
    for layer in cfg["layers"]:
        if layer[0] == "conv":
            _, ci, co, k, s, relu = layer
        else:
            _, ci, k, s = layer
            co, relu = ci, False
        Ho, Wo = hx.hex_out_shape(H, W, k, s)
        out.append((layer[0], ci, co, k, s, relu, H, W, Ho, Wo))
        H, W = Ho, Wo
    return out


def stack_flop(cfg, N):
    """Products per step: forward of every conv, data gradient of every conv
    but the first, weight gradient of every conv."""
    f = 0.0
    for li, (kind, ci, co, k, s, relu, H, W, Ho, Wo) in enumerate(stack_shapes(cfg)):
        if kind == "conv":
            per = conv_flop(N, ci, co, Ho, Wo, hx.hex_num_taps(k))
            f += per * (2 if li == 0 else 3)
    return f


def cpu_baseline_stack(cfg, d, seconds):
    """The fp64 oracle running the whole stack forward and backward on a
    2-image slice, repeated for `seconds`; returns samples/s."""
    import oracle
    n = 2
    shapes = stack_shapes(cfg)
    reps, t0 = 0, time.perf_counter()
    while True:
        acts, ams = [d["x"][:n]], []
        for li, (kind, ci, co, k, s, relu, H, W, Ho, Wo) in enumerate(shapes):
            a = acts[-1]
            if kind == "conv":
                p = d["params"][li]
                y = oracle.conv_fwd(a, p["w"], p["b"], k, s)
                acts.append(np.maximum(y, 0.0) if relu else y)
                ams.append(None)
            else:
                y, am = oracle.pool_fwd(a, k, s, oracle.POOL_MAX)
                acts.append(y)
                ams.append(am)
        g = d["dy"][:n]
        for li in range(len(shapes) - 1, -1, -1):
            kind, ci, co, k, s, relu, H, W, Ho, Wo = shapes[li]
            if kind == "conv":
                oracle.conv_bwd_weight(acts[li], g, k, s)
                if li > 0:
                    g = oracle.conv_bwd_data(g, d["params"][li]["w"], k, s, H, W)
            else:
                relu_y = acts[li] if shapes[li - 1][0] == "conv" and shapes[li - 1][5] else None
                g = oracle.pool_bwd(g, ams[li], relu_y, k, s, oracle.POOL_MAX, H, W)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return n * reps / el, oracle.threads(), reps, el


def bench_stack(args, torch, cfg_key):
    cfg = gen.CONFIGS[cfg_key]
    N = cfg["N"]
    dt = torch.bfloat16
    shapes = stack_shapes(cfg)
    Hl, Wl = shapes[-1][8], shapes[-1][9]
    nsets = 2
    dsets = [gen.stack_inputs(cfg, hx.hex_num_taps, (Hl, Wl), seed=b) for b in range(nsets)]
    params = [None if p is None else dict(w=dev(torch, p["w"], dt), b=dev(torch, p["b"], dt))
              for p in dsets[0]["params"]]
    xs = [dev(torch, d["x"], dt) for d in dsets]
    dys = [dev(torch, d["dy"], dt) for d in dsets]
    acts = []     # output of each layer
    grads = []    # gradient w.r.t. each layer's input (None for the image)
    ams = []
    wgr = []
    nws = 0
    for li, (kind, ci, co, k, s, relu, H, W, Ho, Wo) in enumerate(shapes):
        acts.append(torch.empty((N, co, Ho, Wo), dtype=dt, device="cuda:0"))
        grads.append(None if li == 0 else torch.empty((N, ci, H, W), dtype=dt, device="cuda:0"))
        if kind == "conv":
            T = hx.hex_num_taps(k)
            ams.append(None)
            wgr.append((torch.empty((co, ci, T), dtype=torch.float32, device="cuda:0"),
                        torch.empty((co,), dtype=torch.float32, device="cuda:0")))
            nws = max(nws, hx.hexconv_bwd_workspace(N, ci, co, H, W, k, s, hx.HEX_BF16))
        else:
            ams.append(torch.empty((N, co, Ho, Wo), dtype=torch.uint8, device="cuda:0"))
            wgr.append(None)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda:0")

    def forward(i):
        a = xs[i % nsets]
        for li, (kind, ci, co, k, s, relu, H, W, Ho, Wo) in enumerate(shapes):
            if kind == "conv":
                hx.hexconv_fwd(a, params[li]["w"], params[li]["b"], acts[li], k, s, relu=relu)
            else:
                hx.hexpool_fwd(a, acts[li], ams[li], k, s, hx.HEX_POOL_MAX)
            a = acts[li]

    def backward(i):
        g = dys[i % nsets]
        for li in range(len(shapes) - 1, -1, -1):
            kind, ci, co, k, s, relu, H, W, Ho, Wo = shapes[li]
            a_in = xs[i % nsets] if li == 0 else acts[li - 1]
            if kind == "conv":
                hx.hexconv_bwd(a_in, g, params[li]["w"], grads[li], wgr[li][0], wgr[li][1], ws,
                               k, s)
            else:
                relu_y = a_in if shapes[li - 1][0] == "conv" and shapes[li - 1][5] else None
                hx.hexpool_bwd(g, ams[li], relu_y, grads[li], k, s, hx.HEX_POOL_MAX)
            g = grads[li]

    def step(i):
        forward(i)
        backward(i)

    timer = EagerTimer(torch) if args.eager else GraphTimer(torch)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_step = timer.time(step, args.steps)
    # per-layer durations (each call alone, same inputs every time)
    per_layer = []
    op_fns = {}
    for li, (kind, ci, co, k, s, relu, H, W, Ho, Wo) in enumerate(shapes):
        a_in = xs[0] if li == 0 else acts[li - 1]
        if kind == "conv":
            f = lambda i, li=li, a_in=a_in, k=k, s=s, relu=relu: hx.hexconv_fwd(
                a_in, params[li]["w"], params[li]["b"], acts[li], k, s, relu=relu)
            b = lambda i, li=li, a_in=a_in, k=k, s=s: hx.hexconv_bwd(
                a_in, acts[li], params[li]["w"], grads[li], wgr[li][0], wgr[li][1], ws, k, s)
        else:
            f = lambda i, li=li, a_in=a_in, k=k, s=s: hx.hexpool_fwd(
                a_in, acts[li], ams[li], k, s, hx.HEX_POOL_MAX)
            relu_y = a_in if shapes[li - 1][0] == "conv" and shapes[li - 1][5] else None
            b = lambda i, li=li, k=k, s=s, relu_y=relu_y: hx.hexpool_bwd(
                acts[li], ams[li], relu_y, grads[li], k, s, hx.HEX_POOL_MAX)
        op_fns[(li, "fwd")], op_fns[(li, "bwd")] = f, b
        per_layer.append(dict(layer=li, kind=kind, C_in=ci, C_out=co, k=k, stride=s,
                              fwd_ms=round(timer.time(f, args.steps), 5),
                              bwd_ms=round(timer.time(b, args.steps), 5)))
    flop = stack_flop(cfg, N)
    out = dict(
        metric="hex-CNN stack samples/s (fwd+bwd)", value=round(N / (ms_step * 1e-3), 1),
        unit="samples/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
        ms_per_step=round(ms_step, 5), higher_is_better=True, scaling="weak",
        vs_baseline=None, dtype="bf16", data="synthetic",
        config=dict(workload=cfg["name"], N=N, H=cfg["H"], W=cfg["W"],
                    layers=[list(l) for l in cfg["layers"]]),
        GFLOPs=round(flop / (ms_step * 1e-3) / 1e9, 1),
        per_layer=per_layer,
    )
    # dominant layer op against its roofline
    best = max([(pl["fwd_ms"], li, "fwd") for li, pl in enumerate(per_layer)] +
               [(pl["bwd_ms"], li, "bwd") for li, pl in enumerate(per_layer)])
    ms, li, op = best
    kind, ci, co, k, s, relu, H, W, Ho, Wo = shapes[li]
    kname, kms, kper, kall = dominant_kernel(torch, op_fns[(li, op)], args.steps)
    if kind == "conv" and ci >= 32:
        # products of the op: forward 1, backward 2 (data and weight gradients)
        units = conv_flop(N, ci, co, Ho, Wo, hx.hex_num_taps(k)) * products_of(kname, op) / kper
        ach = units / (kms * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=round(ach, 2), peak=BF16_MFMA_PEAK_TFLOPS,
                    unit="TFLOP/s", frac=round(ach / BF16_MFMA_PEAK_TFLOPS, 4))
    else:
        if kind == "conv":
            nb = 2 * (N * ci * H * W + N * co * Ho * Wo) * (1 if op == "fwd" else 2)
        else:
            nb = 2 * (N * ci * H * W + N * co * Ho * Wo) + N * co * Ho * Wo
        units = nb / kper
        ach = units / (kms * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=round(ach, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(ach / HBM_PEAK_GBS, 4))
    roof["traffic"] = read_counters(cfg["name"], kname)
    roof.update(kernel=kname, kernel_ms=round(kms, 5), launches_per_op=kper,
                op="layer%d_%s" % (li, op), alg_per_launch=units, op_kernels_ms=kall)
    out["roofline"] = roof
    if not args.no_cpu_baseline:
        sps, thr, reps, el = cpu_baseline_stack(cfg, dsets[0], args.cpu_seconds)
        out["cpu_baseline"] = dict(
            value=round(sps, 3), unit="samples/s", cores=thr, kind="oracle",
            sample="2 of %d images through the whole stack, fwd+bwd, fp64, repeated %d "
                   "times in %.1f s" % (N, reps, el))
    return out


def main():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=500)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--config", default="c2", choices=["c1", "c2", "c3", "c4", "c5"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--eager", action="store_true",
                   help="launch eagerly instead of replaying a HIP graph (for counter runs)")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="after the benchmark, one device-to-device copy of this many MiB "
                        "(counter calibration for paper_1903_01814_amd.counters)")
    args = p.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this library runs on a single GPU; --gpus %d is not supported "
              "(the batch would be sharded across GPUs, one process each)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    hx.load()
    if args.config == "c3":
        out = bench_pool(args, torch, args.config)
    elif args.config == "c5":
        out = bench_stack(args, torch, args.config)
    else:
        out = bench_conv(args, torch, args.config)
    print(json.dumps(out), flush=True)
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib << 18                    # float32 elements
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()


if __name__ == "__main__":
    main()
