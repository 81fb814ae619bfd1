"""Seeded synthetic inputs for the five benchmark workloads.

This module only draws random numbers and rounds them to the compute dtype;
it holds none of the convolution or pooling arithmetic.  The same arrays feed
the GPU library and the fp64 reference, so both see identical operand bits.

The workloads mimic imaging-Cherenkov camera data (the application the
HexagDLy paper, arXiv:1903.01814, targets in Sec. 1 and 5): sparse positive
images (log-normal amplitudes times a Bernoulli(0.1) mask) on a hexagonal
camera footprint, plus dense Gaussian activations for the wide layers.  No
real camera data is used.

Every generator draws from ``numpy.random.default_rng(seed)`` in the fixed
order x, mask, w, b, dy; values are drawn in float64, rounded to float32 and,
for bf16 workloads, rounded again (round-to-nearest-even) to bfloat16.  The
returned arrays are float64 holding exactly representable values.
"""
from __future__ import annotations

import math

import numpy as np

F32 = "f32"
BF16 = "bf16"

# The five workloads.  Sizes are the network input sizes H x W; outputs follow
# from the hex-preserving stride.
CONFIGS = {
    "c1": dict(name="c1_tiny_fwd_fp32", kind="conv", N=4, C_in=1, C_out=4,
               H=16, W=16, k=1, stride=1, dtype=F32, bias=True, bwd=False,
               x_dist="uniform"),
    "c2": dict(name="c2_camera_fwd_bwd_fp32", kind="conv", N=256, C_in=1,
               C_out=16, H=40, W=40, k=2, stride=1, dtype=F32, bias=True,
               bwd=True, x_dist="camera_footprint"),
    "c3": dict(name="c3_pool_fwd_bf16", kind="pool", N=256, C=64, H=40, W=40,
               k=1, stride=2, dtype=BF16, x_dist="normal"),
    "c4": dict(name="c4_wide_fwd_bwd_bf16", kind="conv", N=64, C_in=64,
               C_out=64, H=128, W=128, k=1, stride=1, dtype=BF16, bias=True,
               bwd=True, x_dist="normal"),
    "c5": dict(name="c5_stack_fwd_bwd_bf16", kind="stack", N=512, H=48, W=48,
               dtype=BF16, x_dist="camera_full",
               # conv(1->32,k2)+relu, maxpool(k1,s2), conv(32->64,k2),
               # maxpool(k1,s2), conv(64->128,k1)
               layers=[("conv", 1, 32, 2, 1, True), ("pool", 32, 1, 2),
                       ("conv", 32, 64, 2, 1, False), ("pool", 64, 1, 2),
                       ("conv", 64, 128, 1, 1, False)]),
    # time-resolved camera (hexagonal planes, equidistant time samples):
    # 3-D convolution over a window of 3 time slices, forward and backward
    "c6": dict(name="c6_time_resolved_3d_fp32", kind="conv3d", N=64, C_in=1,
               C_out=16, D=32, H=40, W=40, k=1, kz=1, stride=1, stride_z=1,
               dtype=F32, bias=True, bwd=True, x_dist="camera_footprint"),
}

# Hexagonal camera footprint of config 2: every pixel within 18 neighbour
# layers of element (20, 20) (1 + 3*18*19 = 1027 pixels); the rest is blank
# and filled with 0.
FOOTPRINT_CENTRE = (20, 20)
FOOTPRINT_LAYERS = 18


def round_f32(a):
    return np.asarray(a, np.float64).astype(np.float32).astype(np.float64)


def round_bf16(a):
    """float64 -> float32 (RNE) -> bfloat16 (RNE), returned as float64."""
    f = np.ascontiguousarray(np.asarray(a, np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def round_to(a, dtype):
    return round_bf16(a) if dtype == BF16 else round_f32(a)


def camera_footprint(H: int, W: int, centre=FOOTPRINT_CENTRE,
                     layers=FOOTPRINT_LAYERS):
    """Boolean H x W mask of a hexagonal camera outline.

    Uses the physical pixel positions of the offset-column layout (odd
    columns half a pitch lower): a pixel is inside when it lies in the
    regular hexagon whose corners are `layers` pitches from the centre pixel
    along the six neighbour directions.
    """
    r = np.arange(H)[:, None].astype(np.float64)
    c = np.arange(W)[None, :].astype(np.float64)
    cx = c * math.sqrt(3.0) / 2.0
    cy = r + 0.5 * (np.arange(W)[None, :] % 2)
    r0, c0 = centre
    dx = cx - c0 * math.sqrt(3.0) / 2.0
    dy = cy - (r0 + 0.5 * (c0 % 2))
    a = np.abs(2.0 * dx / math.sqrt(3.0))
    b1 = np.abs(dy - dx / math.sqrt(3.0))
    b2 = np.abs(dy + dx / math.sqrt(3.0))
    return np.maximum(np.maximum(a, b1), b2) <= layers + 1e-6


def _draw_x(rng, shape, dist):
    if dist == "uniform":
        return rng.uniform(0.0, 1.0, size=shape)
    if dist == "normal":
        return rng.standard_normal(size=shape)
    if dist in ("camera_footprint", "camera_full"):
        amp = rng.lognormal(mean=0.0, sigma=1.0, size=shape)
        mask = rng.random(size=shape) < 0.1
        x = amp * mask
        if dist == "camera_footprint":
            x = x * camera_footprint(shape[-2], shape[-1])[None, None]
        return x
    raise ValueError(dist)


def _draw_w(rng, C_out, C_in, T, dist):
    if dist == "he":
        std = math.sqrt(2.0 / (C_in * T))
    else:
        std = 0.1
    return rng.normal(0.0, std, size=(C_out, C_in, T))


def conv_inputs(cfg: dict, T: int, out_hw, seed: int = 0,
                N: int | None = None):
    """x, w, b (or None), dy for a convolution workload, rounded to dtype.

    `T` is the kernel's tap count and `out_hw` the output (H, W), both
    supplied by the caller.  `N` overrides the batch (same per-sample
    recipe).  dy is drawn only for workloads with a backward pass.
    """
    rng = np.random.default_rng(seed)
    n = cfg["N"] if N is None else N
    dt = cfg["dtype"]
    x = _draw_x(rng, (n, cfg["C_in"], cfg["H"], cfg["W"]), cfg["x_dist"])
    wdist = "n01" if cfg["x_dist"] == "uniform" else "he"
    w = _draw_w(rng, cfg["C_out"], cfg["C_in"], T, wdist)
    b = rng.normal(0.0, 0.1, size=cfg["C_out"]) if cfg.get("bias") else None
    out = dict(x=round_to(x, dt), w=round_to(w, dt),
               b=None if b is None else round_to(b, dt))
    if cfg.get("bwd"):
        Ho, Wo = out_hw
        dy = rng.standard_normal(size=(n, cfg["C_out"], Ho, Wo))
        out["dy"] = round_to(dy, dt)
    return out


def pool_inputs(cfg: dict, seed: int = 0, N: int | None = None):
    rng = np.random.default_rng(seed)
    n = cfg["N"] if N is None else N
    x = _draw_x(rng, (n, cfg["C"], cfg["H"], cfg["W"]), cfg["x_dist"])
    return dict(x=round_to(x, cfg["dtype"]))


def stack_inputs(cfg: dict, taps_of, out_hw, seed: int = 0,
                 N: int | None = None):
    """Input image, per-conv-layer (w, b), and the upstream gradient of the
    last layer's output.

    `taps_of(k)` gives a kernel's tap count and `out_hw` the (H, W) of the
    last layer's output, both supplied by the caller.
    """
    rng = np.random.default_rng(seed)
    n = cfg["N"] if N is None else N
    dt = cfg["dtype"]
    x = _draw_x(rng, (n, 1, cfg["H"], cfg["W"]), cfg["x_dist"])
    params = []
    C = 1
    for layer in cfg["layers"]:
        if layer[0] == "conv":
            _, ci, co, k, _s, _relu = layer
            w = _draw_w(rng, co, ci, taps_of(k), "he")
            b = rng.normal(0.0, 0.1, size=co)
            params.append(dict(w=round_to(w, dt), b=round_to(b, dt)))
            C = co
        else:
            params.append(None)
    dy = rng.standard_normal(size=(n, C) + tuple(out_hw))
    return dict(x=round_to(x, dt), params=params, dy=round_to(dy, dt))


def conv3d_inputs(cfg: dict, T: int, out_dhw, seed: int = 0, N: int | None = None):
    """x [N][C_in][D][H][W], w [C_out][C_in][2kz+1][T] (He-normal over the
    (2kz+1) T C_in fan-in), b, dy for a 3-D convolution workload, rounded to
    dtype.  Every plane of x follows the camera recipe of `x_dist`."""
    rng = np.random.default_rng(seed)
    n = cfg["N"] if N is None else N
    dt = cfg["dtype"]
    Z = 2 * cfg["kz"] + 1
    x = _draw_x(rng, (n, cfg["C_in"], cfg["D"], cfg["H"], cfg["W"]), cfg["x_dist"])
    w = _draw_w(rng, cfg["C_out"], cfg["C_in"] * Z, T, "he").reshape(cfg["C_out"], cfg["C_in"],
                                                                    Z, T)
    b = rng.normal(0.0, 0.1, size=cfg["C_out"]) if cfg.get("bias") else None
    out = dict(x=round_to(x, dt), w=round_to(w, dt), b=None if b is None else round_to(b, dt))
    if cfg.get("bwd"):
        dy = rng.standard_normal(size=(n, cfg["C_out"]) + tuple(out_dhw))
        out["dy"] = round_to(dy, dt)
    return out
