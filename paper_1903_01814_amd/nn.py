"""PyTorch layers over libhexconv: hexagonal convolution and pooling as
``torch.autograd.Function``s and ``nn.Module``s, so that they drop into
models written with the PyTorch API the way the paper's layers do (Sec. 2.4).

Tensors are NCHW in the offset-column layout of Sec. 2.1 (odd columns shifted
half a pitch down); weights are ``[C_out, C_in, T]`` with T = 1 + 3k(k+1)
taps in the library's canonical order.  Forward and backward are libhexconv
calls through the ``hexconv`` binding: this module allocates their outputs
and workspaces with torch and keeps what the backward needs, nothing else.
Inputs must live on the GPU in float32 or bfloat16, with weights and bias of
the same dtype; weight and bias gradients are computed in float32 and handed
to autograd in the parameter's dtype.
"""
from __future__ import annotations

import math

import torch
from torch import nn

from . import hexconv as hx


def _empty(shape, like, dtype=None):
    return torch.empty(shape, dtype=like.dtype if dtype is None else dtype,
                       device=like.device)


def _relu_backward(gy, y):
    """gy * [y > 0] by the pooling gradient of the one-tap (k = 0, stride 1)
    average pool, whose gradient is its input, masked by relu_y > 0."""
    g = _empty(gy.shape, gy)
    hx.hexpool_bwd(gy, None, y, g, 0, 1, hx.HEX_POOL_AVG)
    return g


class HexConv2dFunction(torch.autograd.Function):
    """y = hexagonal convolution of x with w (+ b), optionally followed by
    ReLU (fused into the forward kernel's epilogue)."""

    @staticmethod
    def forward(ctx, x, w, b, k, stride, relu):
        x = x.contiguous()
        w = w.contiguous()
        b = None if b is None else b.contiguous()
        if w.dtype != x.dtype or (b is not None and b.dtype != x.dtype):
            raise TypeError("hex_conv2d: x, weight and bias must share a dtype")
        N, _, H, W = x.shape
        Ho, Wo = hx.hex_out_shape(H, W, k, stride)
        y = _empty((N, w.shape[0], Ho, Wo), x)
        hx.hexconv_fwd(x, w, b, y, k, stride, relu=relu)
        ctx.save_for_backward(x, w, y if relu else None)
        ctx.k, ctx.stride, ctx.relu = k, stride, relu
        ctx.has_bias = b is not None
        ctx.bias_dtype = None if b is None else b.dtype
        return y

    @staticmethod
    def backward(ctx, gy):
        x, w, y = ctx.saved_tensors
        k, s = ctx.k, ctx.stride
        gy = gy.contiguous()
        if ctx.relu:
            gy = _relu_backward(gy, y)
        need_x, need_w, need_b = ctx.needs_input_grad[:3]
        need_b = need_b and ctx.has_bias
        dx = dw = db = None
        if not (need_w or need_b):
            if need_x:
                dx = _empty(x.shape, x)
                hx.hexconv_bwd_data(gy, w, dx, k, s)
            return dx, None, None, None, None, None
        N, Ci, H, W = x.shape
        Co = w.shape[0]
        dt = hx.HEX_F32 if x.dtype == torch.float32 else hx.HEX_BF16
        dx = _empty(x.shape, x) if need_x else None
        dw = _empty(w.shape, x, torch.float32)
        db = _empty((Co,), x, torch.float32) if ctx.has_bias else None
        nbytes = hx.hexconv_bwd_workspace(N, Ci, Co, H, W, k, s, dt)
        ws = _empty((nbytes,), x, torch.uint8) if nbytes else None
        hx.hexconv_bwd(x, gy, w, dx, dw, db, ws, k, s)
        gw = dw.to(w.dtype) if need_w else None
        gb = db.to(ctx.bias_dtype) if need_b else None
        return dx, gw, gb, None, None, None


class HexPool2dFunction(torch.autograd.Function):
    """y = hexagonal max or average pooling of x; max pooling keeps the
    winning tap of every output (uint8) for its backward."""

    @staticmethod
    def forward(ctx, x, k, stride, mode):
        x = x.contiguous()
        N, C, H, W = x.shape
        Ho, Wo = hx.hex_out_shape(H, W, k, stride)
        y = _empty((N, C, Ho, Wo), x)
        am = _empty(y.shape, x, torch.uint8) if mode == hx.HEX_POOL_MAX else None
        hx.hexpool_fwd(x, y, am, k, stride, mode)
        ctx.save_for_backward(am)
        ctx.k, ctx.stride, ctx.mode, ctx.in_shape = k, stride, mode, x.shape
        return y

    @staticmethod
    def backward(ctx, gy):
        (am,) = ctx.saved_tensors
        if not ctx.needs_input_grad[0]:
            return None, None, None, None
        dx = _empty(ctx.in_shape, gy)
        hx.hexpool_bwd(gy.contiguous(), am, None, dx, ctx.k, ctx.stride, ctx.mode)
        return dx, None, None, None


def hex_conv2d(x, weight, bias=None, kernel_size=1, stride=1, relu=False):
    """Hexagonal convolution (Sec. 2.3) with a caller-supplied kernel:
    weight [C_out, C_in, 1 + 3k(k+1)], bias [C_out] or None."""
    return HexConv2dFunction.apply(x, weight, bias, int(kernel_size), int(stride),
                                   bool(relu))


def hex_max_pool2d(x, kernel_size, stride):
    """Hexagonal max pooling over the size-k hexagon (Sec. 2.4); taps outside
    the tensor take part as zeros."""
    return HexPool2dFunction.apply(x, int(kernel_size), int(stride), hx.HEX_POOL_MAX)


def hex_avg_pool2d(x, kernel_size, stride):
    """Hexagonal average pooling: the sum over the size-k hexagon divided by
    its tap count, taps outside the tensor counting as zeros (Sec. 2.4)."""
    return HexPool2dFunction.apply(x, int(kernel_size), int(stride), hx.HEX_POOL_AVG)


class HexConv2d(nn.Module):
    """Hexagonal convolution layer of size ``kernel_size`` (the hexagon's
    radius k) and ``stride`` (Sec. 2.3).  ``relu`` fuses a ReLU into the
    forward kernel.  ``debug`` sets every kernel element to 1 and drops the
    bias, the layer then summing each hexagonal neighbourhood (Sec. 3); its
    weights take no gradient.  Initial weights and bias are uniform in
    +-1/sqrt(fan_in) with the hexagonal fan-in C_in * T."""

    def __init__(self, in_channels, out_channels, kernel_size=1, stride=1, bias=True,
                 relu=False, debug=False, device=None, dtype=None):
        super().__init__()
        self.in_channels, self.out_channels = int(in_channels), int(out_channels)
        self.kernel_size, self.stride = int(kernel_size), int(stride)
        self.relu, self.debug = bool(relu), bool(debug)
        T = hx.hex_num_taps(self.kernel_size)
        kw = {"device": device, "dtype": dtype}
        self.weight = nn.Parameter(torch.empty((self.out_channels, self.in_channels, T), **kw),
                                   requires_grad=not self.debug)
        if bias and not self.debug:
            self.bias = nn.Parameter(torch.empty((self.out_channels,), **kw))
        else:
            self.register_parameter("bias", None)
        self.reset_parameters()

    def reset_parameters(self):
        with torch.no_grad():
            if self.debug:
                self.weight.fill_(1.0)
                return
            bound = 1.0 / math.sqrt(self.in_channels * self.weight.shape[2])
            self.weight.uniform_(-bound, bound)
            if self.bias is not None:
                self.bias.uniform_(-bound, bound)

    def forward(self, x):
        return hex_conv2d(x, self.weight, self.bias, self.kernel_size, self.stride,
                          self.relu)

    def extra_repr(self):
        return ("%d, %d, kernel_size=%d, stride=%d, bias=%s, relu=%s, debug=%s"
                % (self.in_channels, self.out_channels, self.kernel_size, self.stride,
                   self.bias is not None, self.relu, self.debug))


class HexMaxPool2d(nn.Module):
    """Hexagonal max pooling of size ``kernel_size`` and ``stride``."""

    def __init__(self, kernel_size, stride):
        super().__init__()
        self.kernel_size, self.stride = int(kernel_size), int(stride)

    def forward(self, x):
        return hex_max_pool2d(x, self.kernel_size, self.stride)

    def extra_repr(self):
        return "kernel_size=%d, stride=%d" % (self.kernel_size, self.stride)


class HexAvgPool2d(nn.Module):
    """Hexagonal average pooling of size ``kernel_size`` and ``stride``."""

    def __init__(self, kernel_size, stride):
        super().__init__()
        self.kernel_size, self.stride = int(kernel_size), int(stride)

    def forward(self, x):
        return hex_avg_pool2d(x, self.kernel_size, self.stride)

    def extra_repr(self):
        return "kernel_size=%d, stride=%d" % (self.kernel_size, self.stride)


# ------------------------------------------------------- three dimensions
# Sec. 2.4: hexagonal x-y planes, equidistant samples along z.  Tensors are
# NCDHW; a kernel of size (k, kz) is the size-k hexagon in the plane times
# the 2kz+1 planes around the centre plane; weights [C_out, C_in, 2kz+1, T];
# stride (s, s_z).

def _pair(v):
    if isinstance(v, (tuple, list)):
        a, b = v
        return int(a), int(b)
    return int(v), int(v)


def _relu_backward3d(gy, y):
    """gy * [y > 0] via the gradient of the one-tap 3-D average pool."""
    g = _empty(gy.shape, gy)
    hx.hexpool3d_bwd(gy, None, y, g, 0, 0, 1, 1, hx.HEX_POOL_AVG)
    return g


class HexConv3dFunction(torch.autograd.Function):
    """y = 3-D hexagonal convolution of x with w (+ b), optionally ReLU."""

    @staticmethod
    def forward(ctx, x, w, b, k, kz, stride, stride_z, relu):
        x = x.contiguous()
        w = w.contiguous()
        b = None if b is None else b.contiguous()
        if w.dtype != x.dtype or (b is not None and b.dtype != x.dtype):
            raise TypeError("hex_conv3d: x, weight and bias must share a dtype")
        N, _, D, H, W = x.shape
        Do, Ho, Wo = hx.hex_out_shape3d(D, H, W, k, kz, stride, stride_z)
        y = _empty((N, w.shape[0], Do, Ho, Wo), x)
        hx.hexconv3d_fwd(x, w, b, y, k, kz, stride, stride_z, relu=relu)
        ctx.save_for_backward(x, w, y if relu else None)
        ctx.geom = (k, kz, stride, stride_z)
        ctx.relu, ctx.has_bias = relu, b is not None
        ctx.bias_dtype = None if b is None else b.dtype
        return y

    @staticmethod
    def backward(ctx, gy):
        x, w, y = ctx.saved_tensors
        k, kz, s, sz = ctx.geom
        gy = gy.contiguous()
        if ctx.relu:
            gy = _relu_backward3d(gy, y)
        need_x, need_w, need_b = ctx.needs_input_grad[:3]
        dx = gw = gb = None
        if need_x:
            dx = _empty(x.shape, x)
            hx.hexconv3d_bwd_data(gy, w, dx, k, kz, s, sz)
        if need_w or (need_b and ctx.has_bias):
            N, Ci, D, H, W = x.shape
            Co = w.shape[0]
            dt = hx.HEX_F32 if x.dtype == torch.float32 else hx.HEX_BF16
            dw = _empty(w.shape, x, torch.float32)
            db = _empty((Co,), x, torch.float32) if ctx.has_bias else None
            nbytes = hx.hexconv3d_bwd_weight_workspace(N, Ci, Co, D, H, W, k, kz, s, sz, dt)
            ws = _empty((nbytes,), x, torch.uint8) if nbytes else None
            hx.hexconv3d_bwd_weight(x, gy, dw, db, ws, k, kz, s, sz)
            gw = dw.to(w.dtype) if need_w else None
            gb = db.to(ctx.bias_dtype) if need_b and ctx.has_bias else None
        return dx, gw, gb, None, None, None, None, None


class HexPool3dFunction(torch.autograd.Function):
    """y = 3-D hexagonal max or average pooling; max pooling keeps the
    winning tap (a 16-bit index) for its backward."""

    @staticmethod
    def forward(ctx, x, k, kz, stride, stride_z, mode):
        x = x.contiguous()
        N, C, D, H, W = x.shape
        Do, Ho, Wo = hx.hex_out_shape3d(D, H, W, k, kz, stride, stride_z)
        y = _empty((N, C, Do, Ho, Wo), x)
        am = _empty(y.shape, x, torch.int16) if mode == hx.HEX_POOL_MAX else None
        hx.hexpool3d_fwd(x, y, am, k, kz, stride, stride_z, mode)
        ctx.save_for_backward(am)
        ctx.geom = (k, kz, stride, stride_z)
        ctx.mode, ctx.in_shape = mode, x.shape
        return y

    @staticmethod
    def backward(ctx, gy):
        (am,) = ctx.saved_tensors
        if not ctx.needs_input_grad[0]:
            return None, None, None, None, None, None
        dx = _empty(ctx.in_shape, gy)
        hx.hexpool3d_bwd(gy.contiguous(), am, None, dx, *ctx.geom, ctx.mode)
        return dx, None, None, None, None, None


def hex_conv3d(x, weight, bias=None, kernel_size=(1, 0), stride=(1, 1), relu=False):
    """3-D hexagonal convolution (Sec. 2.4) with a caller-supplied kernel
    weight [C_out, C_in, 2kz+1, 1 + 3k(k+1)]; kernel_size = (k, kz), stride
    = (s, s_z) (an int applies to both)."""
    k, kz = _pair(kernel_size)
    s, sz = _pair(stride)
    return HexConv3dFunction.apply(x, weight, bias, k, kz, s, sz, bool(relu))


def hex_max_pool3d(x, kernel_size, stride):
    """3-D hexagonal max pooling over the (k, kz) window (Sec. 2.4)."""
    k, kz = _pair(kernel_size)
    s, sz = _pair(stride)
    return HexPool3dFunction.apply(x, k, kz, s, sz, hx.HEX_POOL_MAX)


def hex_avg_pool3d(x, kernel_size, stride):
    """3-D hexagonal average pooling over the (k, kz) window (Sec. 2.4)."""
    k, kz = _pair(kernel_size)
    s, sz = _pair(stride)
    return HexPool3dFunction.apply(x, k, kz, s, sz, hx.HEX_POOL_AVG)


class HexConv3d(nn.Module):
    """3-D hexagonal convolution layer: kernel_size = (k, kz), stride = (s,
    s_z); initial weights uniform in +-1/sqrt(C_in (2kz+1) T)."""

    def __init__(self, in_channels, out_channels, kernel_size=(1, 1), stride=(1, 1), bias=True,
                 relu=False, device=None, dtype=None):
        super().__init__()
        self.in_channels, self.out_channels = int(in_channels), int(out_channels)
        self.kernel_size, self.stride = _pair(kernel_size), _pair(stride)
        self.relu = bool(relu)
        k, kz = self.kernel_size
        T = hx.hex_num_taps(k)
        kw = {"device": device, "dtype": dtype}
        self.weight = nn.Parameter(torch.empty((self.out_channels, self.in_channels, 2 * kz + 1, T),
                                               **kw))
        if bias:
            self.bias = nn.Parameter(torch.empty((self.out_channels,), **kw))
        else:
            self.register_parameter("bias", None)
        self.reset_parameters()

    def reset_parameters(self):
        with torch.no_grad():
            fan_in = self.in_channels * self.weight.shape[2] * self.weight.shape[3]
            bound = 1.0 / math.sqrt(fan_in)
            self.weight.uniform_(-bound, bound)
            if self.bias is not None:
                self.bias.uniform_(-bound, bound)

    def forward(self, x):
        return hex_conv3d(x, self.weight, self.bias, self.kernel_size, self.stride, self.relu)

    def extra_repr(self):
        return ("%d, %d, kernel_size=%s, stride=%s, bias=%s, relu=%s"
                % (self.in_channels, self.out_channels, self.kernel_size, self.stride,
                   self.bias is not None, self.relu))


class HexMaxPool3d(nn.Module):
    """3-D hexagonal max pooling, kernel_size = (k, kz), stride = (s, s_z)."""

    def __init__(self, kernel_size, stride):
        super().__init__()
        self.kernel_size, self.stride = _pair(kernel_size), _pair(stride)

    def forward(self, x):
        return hex_max_pool3d(x, self.kernel_size, self.stride)


class HexAvgPool3d(nn.Module):
    """3-D hexagonal average pooling, kernel_size = (k, kz), stride = (s, s_z)."""

    def __init__(self, kernel_size, stride):
        super().__init__()
        self.kernel_size, self.stride = _pair(kernel_size), _pair(stride)

    def forward(self, x):
        return hex_avg_pool3d(x, self.kernel_size, self.stride)
