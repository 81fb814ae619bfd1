#!/usr/bin/env python3
"""Throughput benchmark of libhexconv on one MI355X.

Headline workload (default): the wide-channel hexagonal convolution layer,
bf16 with fp32 accumulation, N=64 images of 128x128, 64 -> 64 channels,
kernel size 1 (7 taps), stride 1 -- the largest of the five workloads
(180 GFLOP per step).  One step = forward, then both gradients (data, and
weight with bias) through the combined backward entry point, over one batch.
Value = effective GFLOP/s counting 2*N*H_out*W_out*C_in*C_out*T for each of
the three products (hex taps only).

Inputs are resident in HBM before timing starts.  The K timed steps are
captured once into a HIP graph and replayed (after W eager warm-up steps and
one untimed replay), so the time is GPU execution, not Python launch cost.
Each step works on a different batch from a rotating set whose total size
exceeds the 256 MB Infinity Cache, so reads and writes go to HBM.  Besides
the mean over the K timed steps, the median (and 10th/90th percentiles) of
at least 50 steps, each replayed and timed on its own, is reported.  A
workload whose one batch fits in the Infinity Cache (c2, c3) also reports
warm_ms_per_step: the same batch every step, so it is served from that
cache; the value is the cold (rotating) figure.

The other workloads are carried as extra keys of the same line ("others"):
c2 (camera-shaped fp32 layer, 1 -> 16 channels, k=2, GFLOP/s), c3 (bf16
max and average pooling, GB/s), c5 (the five-layer bf16 stack, forward
and backward, samples/s) and c6 (3-D convolution of time-resolved camera
data, 32 time slices, 1 -> 16 channels, k=1 over 3 slices, fp32, forward
and backward, GFLOP/s).  --config picks another headline (c1: the tiny
launch-bound forward, reported in microseconds per call).

Prints one JSON line.  With --gpus > 1 it exits: the library runs on one GPU.

--counter-op OP runs only one op of the workload eagerly (--steps times,
after one warm-up step) followed by a device-to-device copy of known size,
and prints nothing timed: the rocprofv3 --pmc passes of
paper_1903_01814_amd.counters run it so that a counter file covers exactly
one op and its kernels.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_1903_01814_amd import hexconv as hx          # noqa: E402
from paper_1903_01814_amd import inputs as gen         # noqa: E402

METRIC = "hex-conv effective GFLOP/s (fwd+bwd) and HBM GB/s vs roofline; samples/s"
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
FP32_PEAK_TFLOPS = 157.3 # fp32 matrix cores and fp32 vector units alike
SIMDS = 1024                      # 256 CUs x 4 SIMDs (MFMA utilisation denominator)
CACHE_BYTES = 256 << 20
ROTATE_MIN_BYTES = 3 * CACHE_BYTES
MEDIAN_REPS = 60


def source_hash():
    h = hashlib.sha1()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_1903_01814_amd", "csrc", "*"))):
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:12]


def counter_file(workload, op, kernel):
    return os.path.join(ROOT, "profiles", "counters_%s_%s_%s.txt" % (workload, op, kernel))


def read_counters(workload, op, kernel):
    """Counters per launch of `kernel` while running `op` of `workload`,
    from the committed rocprofv3 --pmc summary -- only if it was taken on
    the current kernel sources and for exactly this (workload, op, kernel)."""
    path = counter_file(workload, op, kernel)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            a, b = line.split(":", 1)
            kv[a.strip()] = b.strip()
    if (kv.get("source_hash") != source_hash() or kv.get("kernel") != kernel
            or kv.get("op") != op or kv.get("workload") != workload):
        return None
    out = {"instantiation": kv.get("instantiation")}
    for key in ("hbm_bytes_per_launch", "hbm_read_bytes_per_launch",
                "hbm_write_bytes_per_launch", "mfma_util", "mfma_flop_per_launch",
                "lds_insts_per_launch", "lds_bank_conflict_cycles_per_launch",
                "lds_bank_conflict_frac"):
        try:
            out[key] = float(kv[key])
        except (KeyError, ValueError):
            pass
    return out


def log(msg):
    """Progress on stderr (the JSON line alone goes to stdout)."""
    print("bench.py: " + msg, file=sys.stderr, flush=True)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_cores():
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


class EagerTimer:
    """Plain launches bracketed by HIP events on the current stream."""

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
    replay stream, so host-side launch cost is outside the timed region."""

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


def step_distribution(torch, fn, nsets, reps=MEDIAN_REPS):
    """Median, 10th and 90th percentile (ms) of `reps` single steps: one HIP
    graph per rotating input set, replayed round-robin, each replay timed by
    its own event pair."""
    graphs = []
    torch.cuda.synchronize()
    for b in range(nsets):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn(b)
        g.replay()
        graphs.append(g)
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for r in range(reps):
        ev[r][0].record(st)
        graphs[r % nsets].replay()
        ev[r][1].record(st)
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    del graphs
    return dict(median=round(float(np.median(ms)), 5), p10=round(float(np.percentile(ms, 10)), 5),
                p90=round(float(np.percentile(ms, 90)), 5), reps=reps)


def dominant_kernel(torch, fn, reps):
    """The kernel with the largest GPU time over `reps` eager calls of fn,
    timed by the library (a HIP event pair attached to every launch and
    recorded at the kernel's own start and end, on its stream).  Returns (name, ms per launch, launches per
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


def part_of(kernel, op):
    """The part of a convolution op one launch of `kernel` performs: "fwd",
    "bwd" (both gradients), "bwd_data" or "bwd_weight"."""
    if op.endswith("fwd"):
        return "fwd"
    if op in ("bwd_data", "bwd_weight"):
        return op
    if kernel in BOTH_GRADIENT_KERNELS:
        return "bwd"
    return "bwd_weight" if "wgrad" in kernel else "bwd_data"


def conv_flop(N, Ci, Co, Ho, Wo, T):
    return 2.0 * N * Ho * Wo * Ci * Co * T


def dev(torch, a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype).to("cuda:0")


def roofline_entry(bytes_pl, flop_pl, cpeak, kname, kms, kper, op, kall, workload):
    """Roofline of the dominant kernel: its algorithmic bytes and FLOP per
    launch (the part of the op that kernel performs) over its measured
    duration, against HBM and against the matrix-core peak `cpeak` (TFLOP/s,
    for the kernel's dtype).  The roof that binds is the one the kernel is
    closer to (the larger fraction: at its peak it would take longer); the
    other fraction is reported beside it.  Counters are attached when the
    committed summary matches."""
    t = kms * 1e-3
    roofs = {}
    if bytes_pl:
        a = bytes_pl / t / 1e9
        roofs["hbm"] = dict(bound="hbm", achieved=round(a, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                            frac=round(a / HBM_PEAK_GBS, 4), units=bytes_pl)
    if flop_pl:
        a = flop_pl / t / 1e12
        roofs["mfma"] = dict(bound="mfma", achieved=round(a, 2), peak=cpeak, unit="TFLOP/s",
                             frac=round(a / cpeak, 4), units=flop_pl)
    bound = max(roofs, key=lambda b: roofs[b]["frac"])
    roof = dict(roofs[bound])
    units = roof.pop("units")
    for b, r in roofs.items():
        roof["frac_" + b] = r["frac"]
    cnt = read_counters(workload, op, kname)
    roof["traffic"] = None if cnt is None else cnt.get("hbm_bytes_per_launch")
    roof.update(kernel=kname, kernel_ms=round(kms, 5), launches_per_op=kper, op=op,
                alg_per_launch=units, op_kernels_ms=kall)
    if cnt is not None:
        roof["counters"] = cnt
    return roof


def with_cores(fn, cores):
    import oracle
    full = oracle.threads()
    oracle.set_threads(cores)
    try:
        return fn()
    finally:
        oracle.set_threads(full)


def repeat_for(seconds, body):
    reps, t0 = 0, time.perf_counter()
    while True:
        body()
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            return reps, el


def cpu_baseline_conv(cfg, d, k, s, seconds, n_slice, one_core):
    """The fp64 oracle on an n_slice-image slice of the workload (forward and
    both gradients), repeated for `seconds`: GFLOP/s on all host cores and,
    if one_core, on one core."""
    import oracle
    H, W = cfg["H"], cfg["W"]
    Ho, Wo = oracle.out_shape(H, W, s)
    T = oracle.num_taps(k)
    has_bwd = "dy" in d
    x, dy = d["x"][:n_slice], (d["dy"][:n_slice] if has_bwd else None)
    flop = (3 if has_bwd else 1) * conv_flop(n_slice, cfg["C_in"], cfg["C_out"], Ho, Wo, T)

    def body():
        oracle.conv_fwd(x, d["w"], d["b"], k, s)
        if has_bwd:
            oracle.conv_bwd_data(dy, d["w"], k, s, H, W)
            oracle.conv_bwd_weight(x, dy, k, s)

    reps, el = repeat_for(seconds, body)
    out = dict(value=round(flop * reps / el / 1e9, 3), unit="GFLOP/s", cores=oracle.threads(),
               kind="oracle", cpu_model=cpu_model(), host_cores=host_cores(),
               sample="%d of %d images, %s, fp64, repeated %d times in %.1f s"
                      % (n_slice, cfg["N"], "fwd+bwd_data+bwd_weight" if has_bwd else "fwd",
                         reps, el))
    if one_core:
        reps1, el1 = with_cores(lambda: repeat_for(seconds / 3, body), 1)
        out["value_1core"] = round(flop * reps1 / el1 / 1e9, 3)
    return out


def bench_conv(args, torch, cfg_key, headline=True):
    cfg = gen.CONFIGS[cfg_key]
    N, Ci, Co, H, W, k, s = (cfg[n] for n in ("N", "C_in", "C_out", "H", "W", "k", "stride"))
    T = hx.hex_num_taps(k)
    Ho, Wo = hx.hex_out_shape(H, W, k, s)
    dt = torch.float32 if cfg["dtype"] == gen.F32 else torch.bfloat16
    esz = 4 if dt == torch.float32 else 2
    per_set = esz * (N * Ci * H * W * 2 + N * Co * Ho * Wo * 2)
    # enough batches to exceed the Infinity Cache (a tiny launch-bound
    # workload stops at 256)
    nsets = min(256, max(2, -(-ROTATE_MIN_BYTES // per_set)))
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

    op_fns = dict(fwd=fwd, bwd=bwd, bwd_data=bwd_data, bwd_weight=bwd_weight)
    if args.counter_op:
        return run_counter_op(args, torch, step, op_fns)

    timer = EagerTimer(torch) if args.eager else GraphTimer(torch)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_step = timer.time(step, args.steps)
    dist = step_distribution(torch, step, nsets)
    log("%s: %.5f ms per step (%d steps), median %.5f" % (cfg["name"], ms_step, args.steps,
                                                          dist["median"]))
    warm = timer.time(lambda i: step(0), args.steps) if per_set <= CACHE_BYTES else None

    # per-op durations, each op alone over the same rotation; the step uses
    # fwd and bwd, the separate gradient entry points are timed for reference
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
    op_list = ("fwd", "bwd", "bwd_data", "bwd_weight") if has_bwd else ("fwd",)
    reps_op = max(20, min(args.steps, 200))
    for name in op_list:
        ms = timer.time(op_fns[name], reps_op)
        ops[name] = dict(ms=ms, gbs=bytes_alg[name] / (ms * 1e-3) / 1e9)
    flop_op = conv_flop(N, Ci, Co, Ho, Wo, T)
    flop_step = (3 if has_bwd else 1) * flop_op
    bytes_step = bytes_alg["fwd"] + (bytes_alg["bwd"] if has_bwd else 0)
    value = flop_step / (ms_step * 1e-3) / 1e9

    # the dominant op of the step, and within it the kernel with the most
    # GPU time, against its roofline: the op's algorithmic bytes (or
    # products) per launch of that kernel over its measured duration
    dom = max(("fwd", "bwd") if has_bwd else ("fwd",), key=lambda n: ops[n]["ms"])
    kname, kms, kper, kall = dominant_kernel(torch, op_fns[dom], reps_op)
    cpeak = FP32_PEAK_TFLOPS if esz == 4 else BF16_MFMA_PEAK_TFLOPS
    roof = roofline_entry(bytes_alg[part_of(kname, dom)] / kper,
                          products_of(kname, dom) * flop_op / kper, cpeak, kname, kms, kper, dom,
                          kall, cfg["name"])

    out = dict(
        metric=METRIC, value=round(value, 2), unit="GFLOP/s",
        n_gpus=1, steps=args.steps, warmup=args.warmup, ms_per_step=round(ms_step, 5),
        higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="f32" if esz == 4 else "bf16", data="synthetic",
        config=dict(workload=cfg["name"], N=N, C_in=Ci, C_out=Co, H=H, W=W, k=k, stride=s,
                    taps=T, H_out=Ho, W_out=Wo, rotating_batches=nsets,
                    step=("fwd, then dx+dw+db (hexconv_bwd)" if has_bwd else "fwd")),
        hbm_GBps=round(bytes_step / (ms_step * 1e-3) / 1e9, 1),
        samples_per_s=round(N / (ms_step * 1e-3), 1),
        us_per_step=round(ms_step * 1e3, 3),
        step_ms=dist,
        per_op={n: dict(ms=round(v["ms"], 5), alg_GBps=round(v["gbs"], 1),
                        GFLOPs=round(nprod[n] * flop_op / (v["ms"] * 1e-3) / 1e9, 1))
                for n, v in ops.items()},
        roofline=roof,
    )
    if warm is not None:
        out["warm_ms_per_step"] = round(warm, 5)
    if headline and not args.no_cpu_baseline:
        n_slice = min(N, args.cpu_slice if args.cpu_slice else
                      (N if flop_step < 2e9 else max(4, int(N * 2e9 / flop_step))))
        log("cpu baseline")
        out["cpu_baseline"] = cpu_baseline_conv(cfg, d0, k, s, args.cpu_seconds, n_slice,
                                                one_core=cfg_key in ("c1", "c2", "c3"))
    return out


def cpu_baseline_pool(cfg, x, seconds, one_core):
    """The fp64 oracle's max and average pooling on an 8-image slice,
    repeated for `seconds`; GB/s of the same algorithmic bytes."""
    import oracle
    xs = x[:8]
    k, s = cfg["k"], cfg["stride"]
    Ho, Wo = oracle.out_shape(cfg["H"], cfg["W"], s)
    nbytes = 2 * 2 * (xs.size + xs.shape[0] * xs.shape[1] * Ho * Wo)

    def body():
        oracle.pool_fwd(xs, k, s, oracle.POOL_MAX)
        oracle.pool_fwd(xs, k, s, oracle.POOL_AVG)

    reps, el = repeat_for(seconds, body)
    out = dict(value=round(nbytes * reps / el / 1e9, 3), unit="GB/s", cores=oracle.threads(),
               kind="oracle", cpu_model=cpu_model(), host_cores=host_cores(),
               sample="8 of %d images, max and avg pooling, fp64, repeated %d times in %.1f s"
                      % (cfg["N"], reps, el))
    if one_core:
        reps1, el1 = with_cores(lambda: repeat_for(seconds / 3, body), 1)
        out["value_1core"] = round(nbytes * reps1 / el1 / 1e9, 3)
    return out


def bench_pool(args, torch, cfg_key, headline=True):
    cfg = gen.CONFIGS[cfg_key]
    N, C, H, W, k, s = (cfg[n] for n in ("N", "C", "H", "W", "k", "stride"))
    Ho, Wo = hx.hex_out_shape(H, W, k, s)
    dt = torch.bfloat16
    esz = 2
    in_b, out_b = esz * N * C * H * W, esz * N * C * Ho * Wo
    nsets = max(2, -(-ROTATE_MIN_BYTES // (in_b + 2 * out_b)))
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

    op_fns = dict(max=pmax, avg=pavg)
    if args.counter_op:
        return run_counter_op(args, torch, step, op_fns)
    timer = EagerTimer(torch) if args.eager else GraphTimer(torch)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_step = timer.time(step, args.steps)
    dist = step_distribution(torch, step, nsets)
    log("%s: %.5f ms per step (%d steps), median %.5f" % (cfg["name"], ms_step, args.steps,
                                                          dist["median"]))
    warm = (timer.time(lambda i: step(0), args.steps)
            if in_b + 2 * out_b <= CACHE_BYTES else None)
    ops = {}
    reps_op = max(20, min(args.steps, 200))
    for name, fn in op_fns.items():
        ms = timer.time(fn, reps_op)
        ops[name] = dict(ms=ms, gbs=(in_b + out_b) / (ms * 1e-3) / 1e9)
    value = 2 * (in_b + out_b) / (ms_step * 1e-3) / 1e9
    dom = max(ops, key=lambda n: ops[n]["ms"])
    kname, kms, kper, kall = dominant_kernel(torch, op_fns[dom], reps_op)
    roof = roofline_entry((in_b + out_b) / kper, None, None, kname, kms, kper, dom, kall,
                          cfg["name"])
    out = dict(
        metric=METRIC, value=round(value, 1), unit="GB/s",
        n_gpus=1, steps=args.steps, warmup=args.warmup, ms_per_step=round(ms_step, 5),
        higher_is_better=True, scaling="weak", vs_baseline=None, dtype="bf16",
        data="synthetic",
        config=dict(workload=cfg["name"], N=N, C=C, H=H, W=W, k=k, stride=s, H_out=Ho,
                    W_out=Wo, rotating_batches=nsets, step="max pool, then average pool"),
        samples_per_s=round(N / (ms_step * 1e-3), 1),
        step_ms=dist,
        per_op={n: dict(ms=round(v["ms"], 5), alg_GBps=round(v["gbs"], 1))
                for n, v in ops.items()},
        roofline=roof,
    )
    if warm is not None:
        out["warm_ms_per_step"] = round(warm, 5)
    if headline and not args.no_cpu_baseline:
        log("cpu baseline")
        out["cpu_baseline"] = cpu_baseline_pool(cfg, d0["x"], args.cpu_seconds, one_core=True)
    return out


def bench_conv3d(args, torch, cfg_key, headline=True):
    """3-D hexagonal convolution (time-resolved camera): one step = forward,
    then the data and weight gradients, over one batch; GFLOP/s."""
    cfg = gen.CONFIGS[cfg_key]
    N, Ci, Co, D, H, W, k, kz, s, sz = (cfg[n] for n in ("N", "C_in", "C_out", "D", "H", "W",
                                                         "k", "kz", "stride", "stride_z"))
    T = hx.hex_num_taps(k)
    Z = 2 * kz + 1
    Do, Ho, Wo = hx.hex_out_shape3d(D, H, W, k, kz, s, sz)
    dt = torch.float32 if cfg["dtype"] == gen.F32 else torch.bfloat16
    esz = 4 if dt == torch.float32 else 2
    x_b, y_b = esz * N * Ci * D * H * W, esz * N * Co * Do * Ho * Wo
    nsets = max(2, -(-ROTATE_MIN_BYTES // (2 * x_b + 2 * y_b)))
    d0 = gen.conv3d_inputs(cfg, T, (Do, Ho, Wo), seed=0)
    sets = []
    for b in range(nsets):
        d = d0 if b == 0 else gen.conv3d_inputs(cfg, T, (Do, Ho, Wo), seed=b)
        sets.append(dict(x=dev(torch, d["x"], dt), dy=dev(torch, d["dy"], dt),
                         y=torch.empty((N, Co, Do, Ho, Wo), dtype=dt, device="cuda:0"),
                         dx=torch.empty((N, Ci, D, H, W), dtype=dt, device="cuda:0")))
    w = dev(torch, d0["w"], dt)
    bias = dev(torch, d0["b"], dt)
    dw = torch.empty((Co, Ci, Z, T), dtype=torch.float32, device="cuda:0")
    db = torch.empty((Co,), dtype=torch.float32, device="cuda:0")
    nws = hx.hexconv3d_bwd_weight_workspace(N, Ci, Co, D, H, W, k, kz, s, sz,
                                            hx.HEX_F32 if esz == 4 else hx.HEX_BF16)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda:0")

    def fwd(i):
        z = sets[i % nsets]
        hx.hexconv3d_fwd(z["x"], w, bias, z["y"], k, kz, s, sz)

    def bwd_data(i):
        z = sets[i % nsets]
        hx.hexconv3d_bwd_data(z["dy"], w, z["dx"], k, kz, s, sz)

    def bwd_weight(i):
        z = sets[i % nsets]
        hx.hexconv3d_bwd_weight(z["x"], z["dy"], dw, db, ws, k, kz, s, sz)

    def step(i):
        fwd(i)
        bwd_data(i)
        bwd_weight(i)

    op_fns = dict(fwd=fwd, bwd_data=bwd_data, bwd_weight=bwd_weight)
    if args.counter_op:
        return run_counter_op(args, torch, step, op_fns)
    timer = EagerTimer(torch) if args.eager else GraphTimer(torch)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_step = timer.time(step, args.steps)
    dist = step_distribution(torch, step, nsets)
    log("%s: %.5f ms per step (%d steps), median %.5f" % (cfg["name"], ms_step, args.steps,
                                                          dist["median"]))
    g_b = 4 * (Co * Ci * Z * T + Co)
    bytes_alg = {"fwd": x_b + y_b + esz * (Co * Ci * Z * T + Co),
                 "bwd_data": y_b + x_b + esz * Co * Ci * Z * T,
                 "bwd_weight": x_b + y_b + g_b}
    flop_op = 2.0 * N * Do * Ho * Wo * Ci * Co * Z * T
    reps_op = max(20, min(args.steps, 200))
    ops = {}
    for name, fn in op_fns.items():
        ms = timer.time(fn, reps_op)
        ops[name] = dict(ms=ms, gbs=bytes_alg[name] / (ms * 1e-3) / 1e9)
    dom = max(ops, key=lambda n: ops[n]["ms"])
    kname, kms, kper, kall = dominant_kernel(torch, op_fns[dom], reps_op)
    roof = roofline_entry(bytes_alg[part_of(kname, dom)] / kper,
                          flop_op / kper, FP32_PEAK_TFLOPS if esz == 4 else BF16_MFMA_PEAK_TFLOPS,
                          kname, kms, kper, dom, kall, cfg["name"])
    out = dict(
        metric=METRIC, value=round(3 * flop_op / (ms_step * 1e-3) / 1e9, 2), unit="GFLOP/s",
        n_gpus=1, steps=args.steps, warmup=args.warmup, ms_per_step=round(ms_step, 5),
        higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="f32" if esz == 4 else "bf16", data="synthetic",
        config=dict(workload=cfg["name"], N=N, C_in=Ci, C_out=Co, D=D, H=H, W=W, k=k, kz=kz,
                    stride=s, stride_z=sz, taps=Z * T, D_out=Do, H_out=Ho, W_out=Wo,
                    rotating_batches=nsets, step="fwd, then dx, then dw+db"),
        hbm_GBps=round(sum(bytes_alg.values()) / (ms_step * 1e-3) / 1e9, 1),
        samples_per_s=round(N / (ms_step * 1e-3), 1),
        step_ms=dist,
        per_op={n: dict(ms=round(v["ms"], 5), alg_GBps=round(v["gbs"], 1),
                        GFLOPs=round(flop_op / (v["ms"] * 1e-3) / 1e9, 1))
                for n, v in ops.items()},
        roofline=roof,
    )
    if headline and not args.no_cpu_baseline:
        import oracle
        n_slice = 8
        xs, dys = d0["x"][:n_slice], d0["dy"][:n_slice]

        def body():
            oracle.conv3d_fwd(xs, d0["w"], d0["b"], k, kz, s, sz)
            oracle.conv3d_bwd_data(dys, d0["w"], k, kz, s, sz, D, H, W)
            oracle.conv3d_bwd_weight(xs, dys, k, kz, s, sz)

        log("cpu baseline")
        reps, el = repeat_for(args.cpu_seconds, body)
        out["cpu_baseline"] = dict(
            value=round(3 * flop_op * n_slice / N * reps / el / 1e9, 3), unit="GFLOP/s",
            cores=oracle.threads(), kind="oracle", cpu_model=cpu_model(), host_cores=host_cores(),
            sample="%d of %d events, fwd+bwd_data+bwd_weight, fp64, repeated %d times in %.1f s"
                   % (n_slice, N, reps, el))
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

    def body():
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

    reps, el = repeat_for(seconds, body)
    return dict(value=round(n * reps / el, 3), unit="samples/s", cores=oracle.threads(),
                kind="oracle", cpu_model=cpu_model(), host_cores=host_cores(),
                sample="2 of %d images through the whole stack, fwd+bwd, fp64, repeated %d "
                       "times in %.1f s" % (cfg["N"], reps, el))


def bench_stack(args, torch, cfg_key, headline=True):
    cfg = gen.CONFIGS[cfg_key]
    N = cfg["N"]
    dt = torch.bfloat16
    shapes = stack_shapes(cfg)
    Hl, Wl = shapes[-1][8], shapes[-1][9]
    nsets = 3
    dsets = [gen.stack_inputs(cfg, hx.hex_num_taps, (Hl, Wl), seed=b) for b in range(nsets)]
    params = [None if p is None else dict(w=dev(torch, p["w"], dt), b=dev(torch, p["b"], dt))
              for p in dsets[0]["params"]]
    xs = [dev(torch, d["x"], dt) for d in dsets]
    dys = [dev(torch, d["dy"], dt) for d in dsets]
    # activations, input gradients and argmaxes per rotating set
    acts = [[] for _ in range(nsets)]
    grads = [[] for _ in range(nsets)]
    ams = [[] for _ in range(nsets)]
    wgr = []
    nws = 0
    for li, (kind, ci, co, k, s, relu, H, W, Ho, Wo) in enumerate(shapes):
        for b in range(nsets):
            acts[b].append(torch.empty((N, co, Ho, Wo), dtype=dt, device="cuda:0"))
            grads[b].append(None if li == 0 else
                            torch.empty((N, ci, H, W), dtype=dt, device="cuda:0"))
            ams[b].append(torch.empty((N, co, Ho, Wo), dtype=torch.uint8, device="cuda:0")
                          if kind == "pool" else None)
        if kind == "conv":
            T = hx.hex_num_taps(k)
            wgr.append((torch.empty((co, ci, T), dtype=torch.float32, device="cuda:0"),
                        torch.empty((co,), dtype=torch.float32, device="cuda:0")))
            nws = max(nws, hx.hexconv_bwd_workspace(N, ci, co, H, W, k, s, hx.HEX_BF16))
        else:
            wgr.append(None)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda:0")

    def relu_before(li):
        return shapes[li - 1][0] == "conv" and shapes[li - 1][5]

    def layer_fwd(li, b):
        kind, ci, co, k, s, relu, H, W, Ho, Wo = shapes[li]
        a = xs[b] if li == 0 else acts[b][li - 1]
        if kind == "conv":
            hx.hexconv_fwd(a, params[li]["w"], params[li]["b"], acts[b][li], k, s, relu=relu)
        else:
            hx.hexpool_fwd(a, acts[b][li], ams[b][li], k, s, hx.HEX_POOL_MAX)

    def layer_bwd(li, b):
        kind, ci, co, k, s, relu, H, W, Ho, Wo = shapes[li]
        a_in = xs[b] if li == 0 else acts[b][li - 1]
        g = dys[b] if li == len(shapes) - 1 else grads[b][li + 1]
        if kind == "conv":
            hx.hexconv_bwd(a_in, g, params[li]["w"], grads[b][li], wgr[li][0], wgr[li][1], ws,
                           k, s)
        else:
            hx.hexpool_bwd(g, ams[b][li], a_in if relu_before(li) else None, grads[b][li], k, s,
                           hx.HEX_POOL_MAX)

    def step(i):
        b = i % nsets
        for li in range(len(shapes)):
            layer_fwd(li, b)
        for li in range(len(shapes) - 1, -1, -1):
            layer_bwd(li, b)

    op_fns = {}
    for li in range(len(shapes)):
        op_fns["layer%d_fwd" % li] = lambda i, li=li: layer_fwd(li, i % nsets)
        op_fns["layer%d_bwd" % li] = lambda i, li=li: layer_bwd(li, i % nsets)
    if args.counter_op:
        return run_counter_op(args, torch, step, op_fns)

    timer = EagerTimer(torch) if args.eager else GraphTimer(torch)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_step = timer.time(step, args.steps)
    dist = step_distribution(torch, step, nsets)
    log("%s: %.5f ms per step (%d steps), median %.5f" % (cfg["name"], ms_step, args.steps,
                                                          dist["median"]))

    # per-layer ops alone, each over rotating copies of its own operands
    # (at least 768 MB per rotation, so that every call reads HBM)
    per_layer = []
    op_units = {}
    reps_op = max(20, min(args.steps, 200))
    rot_fns = {}
    for li, (kind, ci, co, k, s, relu, H, W, Ho, Wo) in enumerate(shapes):
        in_b, out_b = 2 * N * ci * H * W, 2 * N * co * Ho * Wo
        per_call = 2 * (in_b + out_b)
        R = max(2, -(-ROTATE_MIN_BYTES // per_call))
        a_src = xs[0] if li == 0 else acts[0][li - 1]
        a_in = [a_src.clone() for _ in range(R)]
        y_out = [acts[0][li].clone() for _ in range(R)]
        g_in = [y.clone() for y in y_out]
        dxs = [None if li == 0 else grads[0][li].clone() for _ in range(R)]
        if kind == "conv":
            p = params[li]
            f = lambda i, li=li, k=k, s=s, relu=relu, a_in=a_in, y_out=y_out, p=p: \
                hx.hexconv_fwd(a_in[i % len(a_in)], p["w"], p["b"], y_out[i % len(y_out)], k, s,
                               relu=relu)
            bw = lambda i, li=li, k=k, s=s, a_in=a_in, g_in=g_in, dxs=dxs, p=p: hx.hexconv_bwd(
                a_in[i % len(a_in)], g_in[i % len(g_in)], p["w"], dxs[i % len(dxs)],
                wgr[li][0], wgr[li][1], ws, k, s)
            flop = conv_flop(N, ci, co, Ho, Wo, hx.hex_num_taps(k))
            dx_b = in_b if li > 0 else 0 # layer 0 has no data gradient
            op_units["layer%d_fwd" % li] = (
                {"fwd": in_b + out_b}, flop)
            op_units["layer%d_bwd" % li] = (
                {"bwd": in_b + out_b + dx_b, "bwd_weight": in_b + out_b,
                 "bwd_data": out_b + dx_b}, flop)
        else:
            am_out = [ams[0][li].clone() for _ in range(R)]
            ry = [a.clone() for a in a_in] if relu_before(li) else None
            f = lambda i, k=k, s=s, a_in=a_in, y_out=y_out, am_out=am_out: hx.hexpool_fwd(
                a_in[i % len(a_in)], y_out[i % len(y_out)], am_out[i % len(am_out)], k, s,
                hx.HEX_POOL_MAX)
            bw = lambda i, k=k, s=s, g_in=g_in, am_out=am_out, ry=ry, dxs=dxs: hx.hexpool_bwd(
                g_in[i % len(g_in)], am_out[i % len(am_out)],
                None if ry is None else ry[i % len(ry)], dxs[i % len(dxs)], k, s,
                hx.HEX_POOL_MAX)
            am_b = N * co * Ho * Wo
            op_units["layer%d_fwd" % li] = ({"fwd": in_b + out_b + am_b}, None)
            op_units["layer%d_bwd" % li] = (
                {"bwd": out_b + am_b + in_b + (in_b if ry is not None else 0)}, None)
        rot_fns["layer%d_fwd" % li], rot_fns["layer%d_bwd" % li] = f, bw
        per_layer.append(dict(layer=li, kind=kind, C_in=ci, C_out=co, k=k, stride=s,
                              rotating_copies=R,
                              fwd_ms=round(timer.time(f, reps_op), 5),
                              bwd_ms=round(timer.time(bw, reps_op), 5)))
    # every per-layer op against its roofline (its dominant kernel)
    layer_roof = {}
    for op, fn in rot_fns.items():
        kname, kms, kper, kall = dominant_kernel(torch, fn, reps_op)
        byts, flop = op_units[op]
        # the bytes and products of the part of the op its dominant kernel does
        part = part_of(kname, op) if flop is not None else op.rsplit("_", 1)[1]
        b = byts.get(part, byts.get("bwd", byts.get("fwd")))
        r = roofline_entry(b / kper, None if flop is None else flop * products_of(kname, op) / kper,
                           BF16_MFMA_PEAK_TFLOPS, kname, kms, kper, op, kall, cfg["name"])
        layer_roof[op] = dict(kernel=kname, kernel_ms=r["kernel_ms"], bound=r["bound"],
                              frac=r["frac"], achieved=r["achieved"], unit=r["unit"],
                              traffic=r["traffic"], full=r)
    flop = stack_flop(cfg, N)
    out = dict(
        metric=METRIC, value=round(N / (ms_step * 1e-3), 1),
        unit="samples/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
        ms_per_step=round(ms_step, 5), higher_is_better=True, scaling="weak",
        vs_baseline=None, dtype="bf16", data="synthetic",
        config=dict(workload=cfg["name"], N=N, H=cfg["H"], W=cfg["W"],
                    layers=[list(l) for l in cfg["layers"]], rotating_batches=nsets),
        GFLOPs=round(flop / (ms_step * 1e-3) / 1e9, 1),
        step_ms=dist,
        per_layer=per_layer,
        per_layer_roofline={op: {k: v for k, v in r.items() if k != "full"}
                            for op, r in layer_roof.items()},
    )
    # the dominant layer op (by time) carries the line's roofline entry
    dom = max(layer_roof, key=lambda op: layer_roof[op]["kernel_ms"])
    out["roofline"] = layer_roof[dom]["full"]
    if headline and not args.no_cpu_baseline:
        log("cpu baseline")
        out["cpu_baseline"] = cpu_baseline_stack(cfg, dsets[0], args.cpu_seconds)
    return out


def run_counter_op(args, torch, step, op_fns):
    """--counter-op: one warm-up step, then the op alone, then the
    calibration copy; counters are read per dispatch by rocprofv3."""
    if args.counter_op not in op_fns:
        raise SystemExit("bench.py: unknown op %s (have %s)" % (args.counter_op, sorted(op_fns)))
    step(0)
    torch.cuda.synchronize()
    fn = op_fns[args.counter_op]
    for i in range(args.steps):
        fn(i)
    torch.cuda.synchronize()
    calibration_copy(torch, args.calib_copy_mib)
    return dict(counter_op=args.counter_op, launches=args.steps)


def calibration_copy(torch, mib):
    if mib <= 0:
        return
    n = mib << 18                    # float32 elements
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()


BENCHES = {"c1": bench_conv, "c2": bench_conv, "c3": bench_pool, "c4": bench_conv,
           "c5": bench_stack, "c6": bench_conv3d}


def compact(line):
    """The fields of another workload's line carried inside the headline."""
    keep = ("metric", "value", "unit", "ms_per_step", "warm_ms_per_step", "dtype", "config",
            "step_ms", "samples_per_s", "hbm_GBps", "GFLOPs", "per_op", "per_layer",
            "per_layer_roofline", "roofline")
    return {k: line[k] for k in keep if k in line}


def main():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--config", default="c4", choices=sorted(BENCHES))
    p.add_argument("--also", default="c2,c3,c5,c6",
                   help="comma-separated workloads carried as extra keys ('' for none)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--eager", action="store_true",
                   help="launch eagerly instead of replaying a HIP graph")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--cpu-slice", type=int, default=0,
                   help="images of the CPU baseline's slice (0: picked by size)")
    p.add_argument("--counter-op", default=None,
                   help="run only this op (for rocprofv3 --pmc passes); prints no timing")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="after the run, one device-to-device copy of this many MiB "
                        "(counter calibration for paper_1903_01814_amd.counters)")
    args = p.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this library runs on a single GPU; --gpus %d is not supported "
              "(the batch would be sharded across GPUs, one process each)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    hx.load()
    out = BENCHES[args.config](args, torch, args.config)
    if args.counter_op:
        print(json.dumps(out), flush=True)
        return
    others = [c for c in args.also.split(",") if c and c != args.config]
    if others:
        out["others"] = {}
        for c in others:
            sub = argparse.Namespace(**vars(args))
            sub.steps = min(args.steps, 100)
            sub.warmup = min(args.warmup, 5)
            line = BENCHES[c](sub, torch, c, headline=False)
            out["others"][gen.CONFIGS[c]["name"]] = compact(line)
            torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)
    calibration_copy(torch, args.calib_copy_mib)


if __name__ == "__main__":
    main()
