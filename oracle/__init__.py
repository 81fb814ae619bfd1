"""fp64 CPU reference ("oracle") for hexagonal convolution and pooling.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The GPU library never
imports, links or calls it, and it shares no code with the GPU library: the
C source (hexoracle.c) carries its own geometry, and ``brute`` re-derives the
geometry a third way from physical pixel positions.

The definitions (HexagDLy, arXiv:1903.01814, Sec. 2.1-2.4) are documented in
the header of hexoracle.c.  This module only marshals numpy float64 arrays to
that C code.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hexoracle.c")
_LIB = os.path.join(_HERE, "libhexoracle.so")

POOL_MAX = 0
POOL_AVG = 1

_lib = None


def build(force: bool = True) -> str:
    """Compile hexoracle.c into libhexoracle.so (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared",
               "-Wall", "-Wextra", "-o", tmp, _SRC]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    dp = ctypes.POINTER(ctypes.c_double)
    ip = ctypes.POINTER(ctypes.c_int)
    lp = ctypes.POINTER(ctypes.c_long)
    i = ctypes.c_int
    L = ctypes.c_long
    sig = {
        "oracle_num_taps": [i],
        "oracle_taps": [i, ip, ip],
        "oracle_step": [i, i, i, i, ip, ip],
        "oracle_centre": [i, i, i, ip, ip],
        "oracle_out_shape": [i, i, i, ip, ip],
        "oracle_conv_fwd": [dp, dp, dp, dp, i, i, i, i, i, i, i],
        "oracle_conv_fwd_at": [dp, dp, dp, lp, L, dp, i, i, i, i, i, i, i],
        "oracle_conv_bwd_data": [dp, dp, dp, i, i, i, i, i, i, i],
        "oracle_conv_bwd_data_at": [dp, dp, lp, L, dp, i, i, i, i, i, i, i],
        "oracle_conv_bwd_weight": [dp, dp, dp, dp, i, i, i, i, i, i, i],
        "oracle_conv_bwd_weight_at": [dp, dp, lp, L, dp, i, i, i, i, i, i, i],
        "oracle_pool_fwd": [dp, dp, ip, i, i, i, i, i, i, i],
        "oracle_pool_bwd": [dp, ip, dp, dp, i, i, i, i, i, i, i],
        "oracle_threads": [],
        "oracle_set_threads": [i],
        "oracle_out_shape3d": [i, i, i, i, i, ip, ip, ip],
        "oracle_conv3d_fwd": [dp, dp, dp, dp] + [i] * 10,
        "oracle_conv3d_bwd_data": [dp, dp, dp] + [i] * 10,
        "oracle_conv3d_bwd_weight": [dp, dp, dp, dp] + [i] * 10,
        "oracle_pool3d_fwd": [dp, dp, ip] + [i] * 10,
        "oracle_pool3d_bwd": [dp, ip, dp, dp] + [i] * 10,
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def _d(a):
    if a is None:
        return None
    assert a.dtype == np.float64 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _i(a):
    if a is None:
        return None
    assert a.dtype == np.int32 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int))


def _l(a):
    assert a.dtype == np.int64 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_long))


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle: %s rejected its arguments" % what)


# ---------------------------------------------------------------- geometry

def num_taps(k: int) -> int:
    return _load().oracle_num_taps(k)


def taps(k: int):
    """Axial tap offsets (dq, ds) of a size-k kernel, canonical order."""
    T = num_taps(k)
    dq = np.zeros(T, np.int32)
    ds = np.zeros(T, np.int32)
    _load().oracle_taps(k, _i(dq), _i(ds))
    return dq, ds


def step(r: int, c: int, dq: int, ds: int):
    """Tensor element reached from (r, c) by the axial step (dq, ds)."""
    ro, co = ctypes.c_int(), ctypes.c_int()
    _load().oracle_step(r, c, dq, ds, ctypes.byref(ro), ctypes.byref(co))
    return ro.value, co.value


def centre(i: int, j: int, stride: int):
    """Input element on which output element (i, j) is centred."""
    ro, co = ctypes.c_int(), ctypes.c_int()
    _load().oracle_centre(i, j, stride, ctypes.byref(ro), ctypes.byref(co))
    return ro.value, co.value


def out_shape(H: int, W: int, stride: int):
    ho, wo = ctypes.c_int(), ctypes.c_int()
    _check(_load().oracle_out_shape(H, W, stride, ctypes.byref(ho),
                                    ctypes.byref(wo)), "out_shape")
    return ho.value, wo.value


def threads() -> int:
    return _load().oracle_threads()


def set_threads(n: int) -> None:
    """Threads of the later parallel loops (timing on fewer cores)."""
    _check(_load().oracle_set_threads(n), "set_threads")


# ------------------------------------------------------------- convolution

def conv_fwd(x, w, b, k, stride=1):
    x, w, b = _f64(x), _f64(w), _f64(b)
    N, Ci, H, W = x.shape
    Co = w.shape[0]
    assert w.shape == (Co, Ci, num_taps(k))
    Ho, Wo = out_shape(H, W, stride)
    y = np.empty((N, Co, Ho, Wo), np.float64)
    _check(_load().oracle_conv_fwd(_d(x), _d(w), _d(b), _d(y), N, Ci, Co, H,
                                   W, k, stride), "conv_fwd")
    return y


def conv_fwd_at(x, w, b, k, stride, flat_idx):
    """Selected outputs, flat indices into y[N][C_out][H_out][W_out]."""
    x, w, b = _f64(x), _f64(w), _f64(b)
    N, Ci, H, W = x.shape
    Co = w.shape[0]
    idx = np.ascontiguousarray(flat_idx, np.int64)
    out = np.empty(idx.size, np.float64)
    _check(_load().oracle_conv_fwd_at(_d(x), _d(w), _d(b), _l(idx), idx.size,
                                      _d(out), N, Ci, Co, H, W, k, stride),
           "conv_fwd_at")
    return out


def conv_bwd_data(dy, w, k, stride, H, W):
    dy, w = _f64(dy), _f64(w)
    N, Co, Ho, Wo = dy.shape
    Ci = w.shape[1]
    assert (Ho, Wo) == out_shape(H, W, stride)
    dx = np.empty((N, Ci, H, W), np.float64)
    _check(_load().oracle_conv_bwd_data(_d(dy), _d(w), _d(dx), N, Ci, Co, H,
                                        W, k, stride), "conv_bwd_data")
    return dx


def conv_bwd_data_at(dy, w, k, stride, H, W, flat_idx):
    """Selected elements of dx, flat indices into dx[N][C_in][H][W]."""
    dy, w = _f64(dy), _f64(w)
    N, Co, Ho, Wo = dy.shape
    Ci = w.shape[1]
    idx = np.ascontiguousarray(flat_idx, np.int64)
    out = np.empty(idx.size, np.float64)
    _check(_load().oracle_conv_bwd_data_at(_d(dy), _d(w), _l(idx), idx.size,
                                           _d(out), N, Ci, Co, H, W, k,
                                           stride), "conv_bwd_data_at")
    return out


def conv_bwd_weight(x, dy, k, stride=1):
    x, dy = _f64(x), _f64(dy)
    N, Ci, H, W = x.shape
    Co = dy.shape[1]
    T = num_taps(k)
    dw = np.empty((Co, Ci, T), np.float64)
    db = np.empty(Co, np.float64)
    _check(_load().oracle_conv_bwd_weight(_d(x), _d(dy), _d(dw), _d(db), N,
                                          Ci, Co, H, W, k, stride),
           "conv_bwd_weight")
    return dw, db


def conv_bwd_weight_at(x, dy, k, stride, flat_idx):
    """Selected elements of dw, flat indices into dw[C_out][C_in][T]."""
    x, dy = _f64(x), _f64(dy)
    N, Ci, H, W = x.shape
    Co = dy.shape[1]
    idx = np.ascontiguousarray(flat_idx, np.int64)
    out = np.empty(idx.size, np.float64)
    _check(_load().oracle_conv_bwd_weight_at(_d(x), _d(dy), _l(idx), idx.size,
                                             _d(out), N, Ci, Co, H, W, k,
                                             stride), "conv_bwd_weight_at")
    return out


# ----------------------------------------------------------------- pooling

def pool_fwd(x, k, stride, mode):
    """Returns (y, argmax_tap int32)."""
    x = _f64(x)
    N, C, H, W = x.shape
    Ho, Wo = out_shape(H, W, stride)
    y = np.empty((N, C, Ho, Wo), np.float64)
    am = np.empty((N, C, Ho, Wo), np.int32)
    _check(_load().oracle_pool_fwd(_d(x), _d(y), _i(am), N, C, H, W, k,
                                   stride, mode), "pool_fwd")
    return y, am


def pool_bwd(dy, argmax, relu_y, k, stride, mode, H, W):
    dy = _f64(dy)
    relu_y = _f64(relu_y)
    N, C, Ho, Wo = dy.shape
    am = None if argmax is None else np.ascontiguousarray(argmax, np.int32)
    dx = np.empty((N, C, H, W), np.float64)
    _check(_load().oracle_pool_bwd(_d(dy), _i(am), _d(relu_y), _d(dx), N, C,
                                   H, W, k, stride, mode), "pool_bwd")
    return dx


# -------------------------------------------------------- three dimensions
# x[N][C][D][H][W]; kernel of size (k, kz): the size-k hexagonal window in
# the plane times the planes dz = -kz .. kz; w[C_out][C_in][2kz+1][T];
# plane stride stride_z (hexoracle.c, "three dimensions").

def out_shape3d(D: int, H: int, W: int, stride: int, stride_z: int):
    do, ho, wo = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check(_load().oracle_out_shape3d(D, H, W, stride, stride_z, ctypes.byref(do),
                                      ctypes.byref(ho), ctypes.byref(wo)), "out_shape3d")
    return do.value, ho.value, wo.value


def conv3d_fwd(x, w, b, k, kz, stride=1, stride_z=1):
    x, w, b = _f64(x), _f64(w), _f64(b)
    N, Ci, D, H, W = x.shape
    Co = w.shape[0]
    assert w.shape == (Co, Ci, 2 * kz + 1, num_taps(k))
    Do, Ho, Wo = out_shape3d(D, H, W, stride, stride_z)
    y = np.empty((N, Co, Do, Ho, Wo), np.float64)
    _check(_load().oracle_conv3d_fwd(_d(x), _d(w), _d(b), _d(y), N, Ci, Co, D, H, W, k, kz,
                                     stride, stride_z), "conv3d_fwd")
    return y


def conv3d_bwd_data(dy, w, k, kz, stride, stride_z, D, H, W):
    dy, w = _f64(dy), _f64(w)
    N, Co = dy.shape[:2]
    Ci = w.shape[1]
    assert dy.shape[2:] == out_shape3d(D, H, W, stride, stride_z)
    dx = np.empty((N, Ci, D, H, W), np.float64)
    _check(_load().oracle_conv3d_bwd_data(_d(dy), _d(w), _d(dx), N, Ci, Co, D, H, W, k, kz,
                                          stride, stride_z), "conv3d_bwd_data")
    return dx


def conv3d_bwd_weight(x, dy, k, kz, stride=1, stride_z=1):
    x, dy = _f64(x), _f64(dy)
    N, Ci, D, H, W = x.shape
    Co = dy.shape[1]
    dw = np.empty((Co, Ci, 2 * kz + 1, num_taps(k)), np.float64)
    db = np.empty(Co, np.float64)
    _check(_load().oracle_conv3d_bwd_weight(_d(x), _d(dy), _d(dw), _d(db), N, Ci, Co, D, H,
                                            W, k, kz, stride, stride_z), "conv3d_bwd_weight")
    return dw, db


def pool3d_fwd(x, k, kz, stride, stride_z, mode):
    """Returns (y, argmax int32: (dz + kz) * T + t of the first maximal tap)."""
    x = _f64(x)
    N, C, D, H, W = x.shape
    Do, Ho, Wo = out_shape3d(D, H, W, stride, stride_z)
    y = np.empty((N, C, Do, Ho, Wo), np.float64)
    am = np.empty((N, C, Do, Ho, Wo), np.int32)
    _check(_load().oracle_pool3d_fwd(_d(x), _d(y), _i(am), N, C, D, H, W, k, kz, stride,
                                     stride_z, mode), "pool3d_fwd")
    return y, am


def pool3d_bwd(dy, argmax, relu_y, k, kz, stride, stride_z, mode, D, H, W):
    dy = _f64(dy)
    relu_y = _f64(relu_y)
    N, C = dy.shape[:2]
    am = None if argmax is None else np.ascontiguousarray(argmax, np.int32)
    dx = np.empty((N, C, D, H, W), np.float64)
    _check(_load().oracle_pool3d_bwd(_d(dy), _i(am), _d(relu_y), _d(dx), N, C, D, H, W, k, kz,
                                     stride, stride_z, mode), "pool3d_bwd")
    return dx
