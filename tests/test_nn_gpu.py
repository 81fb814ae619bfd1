"""GPU parity of the autograd layers (paper_1903_01814_amd.nn) against the
fp64 oracle: forward outputs and every gradient autograd hands back, for
convolution (with and without the fused ReLU and bias, strides 1 and 2, the
small-channel and the wide bf16 paths), both poolings, and a three-layer
stack run as an nn.Sequential.  Same tolerances as the direct ABI tests.
"""
import numpy as np
import pytest

import oracle
from paper_1903_01814_amd import hexconv as hx
from paper_1903_01814_amd import inputs as gen

from gpu_helpers import (bf16_ulp, check, from_dev, round_bf16_f64, to_dev,
                         torch_mod)

pytestmark = pytest.mark.gpu


def _draw(rng, shape, dt, scale=1.0):
    return gen.round_to(rng.normal(size=shape) * scale, dt)


def _param(a, dt):
    return torch_mod().nn.Parameter(to_dev(a, dt))


def _leaf(a, dt):
    return to_dev(a, dt).requires_grad_(True)


def _check_conv_grads(x, w, b, g, k, s, dt, xg, wg, bg, what):
    """x.grad, w.grad, b.grad against the oracle for upstream gradient g
    (already masked by the ReLU where there is one)."""
    H, W = x.shape[2:]
    ref = oracle.conv_bwd_data(g, w, k, s, H, W)
    mag = oracle.conv_bwd_data(np.abs(g), np.abs(w), k, s, H, W)
    check(dt, from_dev(xg), ref, mag, what + " dx")
    rw, rb = oracle.conv_bwd_weight(x, g, k, s)
    mw, mb = oracle.conv_bwd_weight(np.abs(x), np.abs(g), k, s)
    check(dt, from_dev(wg), rw, mw, what + " dw")
    if b is not None:
        check(dt, from_dev(bg), rb, mb, what + " db")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", [
    # N, C_in, C_out, H, W, k, stride, bias, relu
    (2, 1, 4, 11, 13, 1, 1, True, False),
    (2, 3, 5, 12, 9, 2, 1, True, True),
    (3, 2, 6, 17, 14, 1, 2, False, True),
    (1, 4, 3, 9, 10, 2, 2, True, False),
    (2, 32, 32, 18, 16, 1, 1, True, True),   # wide channels
    (2, 64, 64, 10, 32, 1, 1, False, False),
])
def test_hexconv2d_autograd(case, dt):
    torch = torch_mod()
    hn = pytest.importorskip("paper_1903_01814_amd.nn")
    N, Ci, Co, H, W, k, s, bias, relu = case
    T = oracle.num_taps(k)
    Ho, Wo = oracle.out_shape(H, W, s)
    rng = np.random.default_rng(sum(case[:7]))
    x = _draw(rng, (N, Ci, H, W), dt)
    w = _draw(rng, (Co, Ci, T), dt, 0.3)
    b = _draw(rng, (Co,), dt, 0.1) if bias else None
    gy = _draw(rng, (N, Co, Ho, Wo), dt)

    layer = hn.HexConv2d(Ci, Co, k, s, bias=bias, relu=relu, device="cuda:0",
                         dtype=torch.float32 if dt == "f32" else torch.bfloat16)
    with torch.no_grad():
        layer.weight.copy_(to_dev(w, dt))
        if bias:
            layer.bias.copy_(to_dev(b, dt))
    xd = _leaf(x, dt)
    y = layer(xd)
    y.backward(to_dev(gy, dt))
    torch.cuda.synchronize()

    yv = from_dev(y)
    ref = oracle.conv_fwd(x, w, b, k, s)
    mag = oracle.conv_fwd(np.abs(x), np.abs(w), None if b is None else np.abs(b), k, s)
    if relu:
        ref = np.maximum(ref, 0.0)
    check(dt, yv, ref, mag, "y")
    # the ReLU's gradient follows the layer's own output (its sign decides)
    g = gy * (yv > 0) if relu else gy
    assert layer.weight.grad.dtype == layer.weight.dtype
    _check_conv_grads(x, w, b, g, k, s, dt, xd.grad, layer.weight.grad,
                      None if b is None else layer.bias.grad, "conv")


def test_hexconv2d_grad_subsets():
    """Only the gradients asked for are computed: input only (data-gradient
    call), weights only (no dx), and a frozen debug layer."""
    torch = torch_mod()
    hn = pytest.importorskip("paper_1903_01814_amd.nn")
    rng = np.random.default_rng(5)
    N, Ci, Co, H, W, k = 2, 3, 4, 10, 12, 1
    x = _draw(rng, (N, Ci, H, W), "f32")
    w = _draw(rng, (Co, Ci, oracle.num_taps(k)), "f32", 0.3)
    gy = _draw(rng, (N, Co, H, W), "f32")
    xd = _leaf(x, "f32")
    wd = to_dev(w, "f32")          # constant kernel (custom values)
    y = hn.hex_conv2d(xd, wd, None, k, 1)
    y.backward(to_dev(gy, "f32"))
    ref = oracle.conv_bwd_data(gy, w, k, 1, H, W)
    check("f32", from_dev(xd.grad), ref, None, "dx only")

    wp = _param(w, "f32")
    y = hn.hex_conv2d(to_dev(x, "f32"), wp, None, k, 1)
    y.backward(to_dev(gy, "f32"))
    rw, _ = oracle.conv_bwd_weight(x, gy, k, 1)
    check("f32", from_dev(wp.grad), rw, None, "dw only")

    # debug layer: all-ones kernel, no bias, no weight gradient; the output
    # is the sum over each in-grid hexagonal neighbourhood
    dbg = hn.HexConv2d(Ci, 1, 2, debug=True, device="cuda:0")
    assert dbg.bias is None and not dbg.weight.requires_grad
    xd = _leaf(x, "f32")
    y = dbg(xd)
    y.sum().backward()
    torch.cuda.synchronize()
    ones = np.ones((1, Ci, oracle.num_taps(2)))
    check("f32", from_dev(y), oracle.conv_fwd(x, ones, None, 2, 1), None, "debug y")
    cnt = from_dev(dbg(torch.ones_like(xd)))
    T2 = oracle.num_taps(2)
    assert np.all(cnt[:, :, 2:-2, 2:-2] == Ci * T2)   # interior: every tap in-grid
    assert np.all(cnt <= Ci * T2) and np.all(cnt >= Ci)
    ref = oracle.conv_bwd_data(np.ones((N, 1, H, W)), ones, 2, 1, H, W)
    check("f32", from_dev(xd.grad), ref, None, "debug dx")
    assert dbg.weight.grad is None


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("mode", [hx.HEX_POOL_MAX, hx.HEX_POOL_AVG])
@pytest.mark.parametrize("case", [(2, 3, 11, 12, 1, 2), (1, 4, 16, 16, 2, 1),
                                  (2, 5, 24, 24, 1, 2), (1, 2, 9, 7, 0, 1),
                                  (2, 3, 24, 32, 3, 2)])
def test_hexpool2d_autograd(case, mode, dt):
    torch = torch_mod()
    hn = pytest.importorskip("paper_1903_01814_amd.nn")
    N, C, H, W, k, s = case
    Ho, Wo = oracle.out_shape(H, W, s)
    rng = np.random.default_rng(sum(case) + 7 * mode)
    x = _draw(rng, (N, C, H, W), dt)
    x[0, 0, : H // 2, : W // 2] = 0.25             # ties
    gy = _draw(rng, (N, C, Ho, Wo), dt)
    pool = (hn.HexMaxPool2d if mode == hx.HEX_POOL_MAX else hn.HexAvgPool2d)(k, s)
    xd = _leaf(x, dt)
    y = pool(xd)
    y.backward(to_dev(gy, dt))
    torch.cuda.synchronize()
    ref, am = oracle.pool_fwd(x, k, s, mode)
    if mode == hx.HEX_POOL_MAX:
        np.testing.assert_array_equal(from_dev(y), ref)
    elif dt == "bf16":
        want = round_bf16_f64(ref)
        assert np.all(np.abs(from_dev(y) - want) <= bf16_ulp(want))
    else:
        check("f32", from_dev(y), ref, None, "avg y")
    amo = am if mode == hx.HEX_POOL_MAX else None
    rdx = oracle.pool_bwd(gy, amo, None, k, s, mode, H, W)
    mag = oracle.pool_bwd(np.abs(gy), amo, None, k, s, mode, H, W)
    check(dt, from_dev(xd.grad), rdx, mag, "pool dx")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_sequential_stack(dt):
    """conv(ReLU) -> max pool -> conv as an nn.Sequential, checked layer by
    layer with each layer's oracle fed the GPU's own activations and
    upstream gradients (a bf16 rounding must not move a pooling winner)."""
    torch = torch_mod()
    hn = pytest.importorskip("paper_1903_01814_amd.nn")
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    rng = np.random.default_rng(11)
    N, H, W = 4, 24, 24
    net = torch.nn.Sequential(
        hn.HexConv2d(1, 16, 2, relu=True, device="cuda:0", dtype=tdt),
        hn.HexMaxPool2d(1, 2),
        hn.HexConv2d(16, 32, 1, device="cuda:0", dtype=tdt))
    c1, pool, c2 = net
    with torch.no_grad():
        for m in (c1, c2):
            m.weight.copy_(to_dev(_draw(rng, tuple(m.weight.shape), dt, 0.3), dt))
            m.bias.copy_(to_dev(_draw(rng, tuple(m.bias.shape), dt, 0.1), dt))
    x = np.abs(_draw(rng, (N, 1, H, W), dt))
    xd = _leaf(x, dt)
    a1 = c1(xd)
    a1.retain_grad()
    a2 = pool(a1)
    a2.retain_grad()
    y = c2(a2)
    gy = _draw(rng, tuple(y.shape), dt)
    y.backward(to_dev(gy, dt))
    torch.cuda.synchronize()

    w1, b1 = from_dev(c1.weight), from_dev(c1.bias)
    w2, b2 = from_dev(c2.weight), from_dev(c2.bias)
    A1, A2 = from_dev(a1), from_dev(a2)
    # forward, layer by layer
    ref = np.maximum(oracle.conv_fwd(x, w1, b1, 2, 1), 0.0)
    mag = oracle.conv_fwd(np.abs(x), np.abs(w1), np.abs(b1), 2, 1)
    check(dt, A1, ref, mag, "stack a1")
    rp, am = oracle.pool_fwd(A1, 1, 2, hx.HEX_POOL_MAX)
    np.testing.assert_array_equal(A2, rp)
    ref = oracle.conv_fwd(A2, w2, b2, 1, 1)
    mag = oracle.conv_fwd(np.abs(A2), np.abs(w2), np.abs(b2), 1, 1)
    check(dt, from_dev(y), ref, mag, "stack y")
    # backward, layer by layer
    _check_conv_grads(A2, w2, b2, gy, 1, 1, dt, a2.grad, c2.weight.grad, c2.bias.grad,
                      "stack conv2")
    G2 = from_dev(a2.grad)
    rdx = oracle.pool_bwd(G2, am, None, 1, 2, hx.HEX_POOL_MAX, H, W)
    mag = oracle.pool_bwd(np.abs(G2), am, None, 1, 2, hx.HEX_POOL_MAX, H, W)
    check(dt, from_dev(a1.grad), rdx, mag, "stack pool dx")
    G1 = from_dev(a1.grad) * (A1 > 0)
    _check_conv_grads(x, w1, b1, G1, 2, 1, dt, xd.grad, c1.weight.grad, c1.bias.grad,
                      "stack conv1")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", [
    # N, C_in, C_out, D, H, W, k, kz, s, sz, bias, relu
    (2, 1, 4, 5, 11, 12, 1, 1, 1, 1, True, False),
    (1, 3, 5, 6, 9, 10, 2, 1, 2, 2, True, True),
    (2, 2, 3, 4, 8, 8, 1, 2, 1, 3, False, True),
])
def test_hexconv3d_autograd(case, dt):
    """HexConv3d forward and every gradient against the 3-D oracle."""
    torch = torch_mod()
    hn = pytest.importorskip("paper_1903_01814_amd.nn")
    N, Ci, Co, D, H, W, k, kz, s, sz, bias, relu = case
    rng = np.random.default_rng(sum(case[:10]))
    T = oracle.num_taps(k)
    x = _draw(rng, (N, Ci, D, H, W), dt)
    layer = hn.HexConv3d(Ci, Co, (k, kz), (s, sz), bias=bias, relu=relu,
                         device="cuda:0", dtype=torch.float32 if dt == "f32" else torch.bfloat16)
    w = from_dev(layer.weight)
    b = from_dev(layer.bias) if bias else None
    xt = _leaf(x, dt)
    y = layer(xt)
    ref = oracle.conv3d_fwd(x, w, b, k, kz, s, sz)
    mag = oracle.conv3d_fwd(np.abs(x), np.abs(w), None if b is None else np.abs(b), k, kz, s, sz)
    if relu:
        ref = np.maximum(ref, 0.0)
    check(dt, from_dev(y), ref, mag, "3d fwd")
    g = _draw(rng, y.shape, dt)
    y.backward(to_dev(g, dt))
    gm = np.where(from_dev(y) > 0, g, 0.0) if relu else g
    check(dt, from_dev(xt.grad), oracle.conv3d_bwd_data(gm, w, k, kz, s, sz, D, H, W),
          oracle.conv3d_bwd_data(np.abs(gm), np.abs(w), k, kz, s, sz, D, H, W), "3d dx")
    rw, rb = oracle.conv3d_bwd_weight(x, gm, k, kz, s, sz)
    mw, mb = oracle.conv3d_bwd_weight(np.abs(x), np.abs(gm), k, kz, s, sz)
    check(dt, from_dev(layer.weight.grad), rw, mw, "3d dw")
    if bias:
        check(dt, from_dev(layer.bias.grad), rb, mb, "3d db")


@pytest.mark.parametrize("mode", ["max", "avg"])
def test_hexpool3d_autograd(mode):
    torch = torch_mod()
    hn = pytest.importorskip("paper_1903_01814_amd.nn")
    rng = np.random.default_rng(3 + (mode == "max"))
    N, C, D, H, W, k, kz, s, sz = 2, 3, 6, 10, 12, 1, 1, 2, 2
    x = _draw(rng, (N, C, D, H, W), "f32")
    pool = (hn.HexMaxPool3d if mode == "max" else hn.HexAvgPool3d)((k, kz), (s, sz))
    xt = _leaf(x, "f32")
    y = pool(xt)
    m = oracle.POOL_MAX if mode == "max" else oracle.POOL_AVG
    ref, am = oracle.pool3d_fwd(x, k, kz, s, sz, m)
    check("f32", from_dev(y), ref, None, "pool3d fwd")
    g = _draw(rng, y.shape, "f32")
    y.backward(to_dev(g, "f32"))
    rdx = oracle.pool3d_bwd(g, am if mode == "max" else None, None, k, kz, s, sz, m, D, H, W)
    check("f32", from_dev(xt.grad), rdx, None, "pool3d dx")
