"""Python binding of libhexconv (include/hexconv.h).

Argument marshalling only: every function has the name of the C entry point
it calls, takes torch tensors for device buffers (torch supplies device
memory and the current HIP stream), checks dtypes/shapes/contiguity, and
raises HexError when the library returns a non-zero status.  All arithmetic
happens in the HIP kernels of libhexconv.so; there is no fallback.  If the
shared library has not been built, loading fails with an error.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhexconv.so")

HEX_OK = 0
HEX_ERR_INVALID_ARG = -1
HEX_ERR_UNSUPPORTED = -2
HEX_ERR_LAUNCH = -3
HEX_F32 = 0
HEX_BF16 = 1
HEX_POOL_MAX = 0
HEX_POOL_AVG = 1
HEX_FLAG_RELU = 1
HEX_MAX_K = 8
HEX_MAX_STRIDE = 8
HEX_MAX_KZ = 4

# (name, argtypes, restype) of every exported symbol
_P = ctypes.c_void_p
_I = ctypes.c_int
_IP = ctypes.POINTER(ctypes.c_int)
_S = ctypes.c_size_t
SIGNATURES = {
    "hex_num_taps": ([_I], _I),
    "hex_out_shape": ([_I, _I, _I, _I, _IP, _IP], _I),
    "hex_tap_table": ([_I, _I, _IP, _IP], _I),
    "hexconv_fwd": ([_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P], _I),
    "hexconv_bwd_data": ([_P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P], _I),
    "hexconv_bwd_weight_workspace": ([_I, _I, _I, _I, _I, _I, _I, _I], _S),
    "hexconv_bwd_weight": ([_P, _P, _P, _P, _P, _S, _I, _I, _I, _I, _I, _I, _I,
                            _I, _P], _I),
    "hexconv_bwd_workspace": ([_I, _I, _I, _I, _I, _I, _I, _I], _S),
    "hexconv_bwd": ([_P, _P, _P, _P, _P, _P, _P, _S, _I, _I, _I, _I, _I, _I, _I,
                     _I, _P], _I),
    "hexconv_bwd_noalloc": ([_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P],
                            _I),
    "hexpool_fwd": ([_P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P], _I),
    "hexpool_bwd": ([_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P], _I),
    "hex_status_string": ([_I], ctypes.c_char_p),
    "hex_last_launch_error": ([], ctypes.c_char_p),
    "hex_out_shape3d": ([_I] * 7 + [_IP, _IP, _IP], _I),
    "hexconv3d_fwd": ([_P, _P, _P, _P] + [_I] * 12 + [_P], _I),
    "hexconv3d_bwd_data": ([_P, _P, _P] + [_I] * 11 + [_P], _I),
    "hexconv3d_bwd_weight_workspace": ([_I] * 11, _S),
    "hexconv3d_bwd_weight": ([_P, _P, _P, _P, _P, _S] + [_I] * 11 + [_P], _I),
    "hexpool3d_fwd": ([_P, _P, _P] + [_I] * 11 + [_P], _I),
    "hexpool3d_bwd": ([_P, _P, _P, _P] + [_I] * 11 + [_P], _I),
    "hexconv_timing_begin": ([], _I),
    "hexconv_timing_end": ([_I, ctypes.c_char_p, _IP, ctypes.POINTER(ctypes.c_double), _IP],
                           _I),
}

HEX_TIMING_NAME_LEN = 64

_lib = None


class HexError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        msg = "%s: %s" % (fn, status_string(status))
        if status == HEX_ERR_LAUNCH:
            msg += " (%s)" % load().hex_last_launch_error().decode()
        super().__init__(msg)


def load():
    """Load libhexconv.so (must have been built, e.g. by build.build()).

    torch is imported first.  torch ships its own HIP runtime (needed under
    the name libamdhip64.so), while libhexconv links the system one
    (libamdhip64.so.7); both then share the HSA runtime that was loaded
    first.  With libhexconv loaded before torch, torch's HIP runtime ends up
    on the system HSA runtime and the system HIP runtime, initialised after
    it, finds no device.  Loading torch's libraries first keeps the one
    order that works."""
    global _lib
    if _lib is None:
        import torch  # noqa: F401  (load order of the HIP runtimes, above)
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                "libhexconv.so not found at %s: build it first "
                "(python -m paper_1903_01814_amd.build)" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            f = getattr(lib, name)
            f.argtypes = args
            f.restype = res
        _lib = lib
    return _lib


def status_string(status: int) -> str:
    return load().hex_status_string(status).decode()


def _ok(fn, rc):
    if rc != HEX_OK:
        raise HexError(fn, rc)


# ----------------------------------------------------------- host helpers

def hex_num_taps(k: int) -> int:
    rc = load().hex_num_taps(k)
    if rc < 0:
        raise HexError("hex_num_taps", rc)
    return rc


def hex_out_shape(H: int, W: int, k: int, stride: int):
    ho, wo = ctypes.c_int(), ctypes.c_int()
    _ok("hex_out_shape", load().hex_out_shape(H, W, k, stride, ctypes.byref(ho),
                                              ctypes.byref(wo)))
    return ho.value, wo.value


def hexconv_timing_begin():
    """Start bracketing every kernel launch with HIP events (eager use only,
    not while a HIP graph is being captured)."""
    _ok("hexconv_timing_begin", load().hexconv_timing_begin())


def hexconv_timing_end(max_kernels: int = 32):
    """Stop recording; {kernel name: (launches, summed GPU ms)} in order of
    first launch."""
    names = ctypes.create_string_buffer(max_kernels * HEX_TIMING_NAME_LEN)
    counts = (ctypes.c_int * max_kernels)()
    total = (ctypes.c_double * max_kernels)()
    n = ctypes.c_int()
    _ok("hexconv_timing_end", load().hexconv_timing_end(max_kernels, names, counts, total,
                                                        ctypes.byref(n)))
    out = {}
    for i in range(n.value):
        raw = names.raw[i * HEX_TIMING_NAME_LEN:(i + 1) * HEX_TIMING_NAME_LEN]
        out[raw.split(b"\0", 1)[0].decode()] = (counts[i], total[i])
    return out


def hex_tap_table(k: int, parity: int):
    """(dcol, drow) lists of the taps of a size-k kernel for a centre column
    of the given parity."""
    T = hex_num_taps(k)
    dcol = (ctypes.c_int * T)()
    drow = (ctypes.c_int * T)()
    _ok("hex_tap_table", load().hex_tap_table(k, parity, dcol, drow))
    return list(dcol), list(drow)


# --------------------------------------------------------- device entries

def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return HEX_F32
    if t.dtype == torch.bfloat16:
        return HEX_BF16
    raise TypeError("hexconv: unsupported dtype %s" % t.dtype)


def _dev(t, name, dt=None, shape=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("hexconv: %s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("hexconv: %s must be contiguous" % name)
    if dt is not None and _dtype_code(t) != dt:
        raise TypeError("hexconv: %s has dtype %s" % (name, t.dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("hexconv: %s has shape %s, expected %s"
                         % (name, tuple(t.shape), tuple(shape)))
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return _torch().cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def hexconv_fwd(x, w, bias, y, k: int, stride: int = 1, relu: bool = False,
                stream=None):
    """y <- hexagonal convolution of x with w (+ bias) (Sec. 2.3)."""
    N, Ci, H, W = x.shape
    Co = w.shape[0]
    dt = _dtype_code(x)
    T = hex_num_taps(k)
    Ho, Wo = hex_out_shape(H, W, k, stride)
    rc = load().hexconv_fwd(
        _dev(x, "x", dt), _dev(w, "w", dt, (Co, Ci, T)),
        _dev(bias, "bias", dt, (Co,)), _dev(y, "y", dt, (N, Co, Ho, Wo)),
        N, Ci, Co, H, W, k, stride, dt, HEX_FLAG_RELU if relu else 0,
        _stream(stream))
    _ok("hexconv_fwd", rc)
    return y


def hexconv_bwd_data(dy, w, dx, k: int, stride: int = 1, stream=None):
    """dx <- gradient of the forward map with respect to its input."""
    N, Ci, H, W = dx.shape
    Co = w.shape[0]
    dt = _dtype_code(dx)
    T = hex_num_taps(k)
    Ho, Wo = hex_out_shape(H, W, k, stride)
    rc = load().hexconv_bwd_data(
        _dev(dy, "dy", dt, (N, Co, Ho, Wo)), _dev(w, "w", dt, (Co, Ci, T)),
        _dev(dx, "dx", dt), N, Ci, Co, H, W, k, stride, dt, _stream(stream))
    _ok("hexconv_bwd_data", rc)
    return dx


def hexconv_bwd_weight_workspace(N, C_in, C_out, H, W, k, stride, dt):
    return load().hexconv_bwd_weight_workspace(N, C_in, C_out, H, W, k, stride,
                                               dt)


def hexconv_bwd_weight(x, dy, dw, db, ws, k: int, stride: int = 1,
                       stream=None):
    """dw, db <- gradients with respect to weights and bias (fp32).  ws is a
    uint8 device tensor of at least hexconv_bwd_weight_workspace bytes (or
    None when that is 0)."""
    torch = _torch()
    N, Ci, H, W = x.shape
    Co = dw.shape[0]
    dt = _dtype_code(x)
    T = hex_num_taps(k)
    Ho, Wo = hex_out_shape(H, W, k, stride)
    if dw.dtype != torch.float32 or (db is not None and db.dtype != torch.float32):
        raise TypeError("hexconv: dw and db must be float32")
    ws_ptr = _dev(ws, "ws")
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    rc = load().hexconv_bwd_weight(
        _dev(x, "x", dt), _dev(dy, "dy", dt, (N, Co, Ho, Wo)),
        _dev(dw, "dw", None, (Co, Ci, T)), _dev(db, "db", None, (Co,)),
        ws_ptr, ws_bytes, N, Ci, Co, H, W, k, stride, dt, _stream(stream))
    _ok("hexconv_bwd_weight", rc)
    return dw, db


def hexconv_bwd_workspace(N, C_in, C_out, H, W, k, stride, dt):
    return load().hexconv_bwd_workspace(N, C_in, C_out, H, W, k, stride, dt)


def hexconv_bwd(x, dy, w, dx, dw, db, ws, k: int, stride: int = 1,
                stream=None):
    """dx (may be None), dw, db (may be None) <- both gradients of one layer
    in one call.  ws: uint8 device tensor of at least hexconv_bwd_workspace
    bytes (or None when that is 0)."""
    torch = _torch()
    N, Ci, H, W = x.shape
    Co = dw.shape[0]
    dt = _dtype_code(x)
    T = hex_num_taps(k)
    Ho, Wo = hex_out_shape(H, W, k, stride)
    if dw.dtype != torch.float32 or (db is not None and db.dtype != torch.float32):
        raise TypeError("hexconv: dw and db must be float32")
    ws_ptr = _dev(ws, "ws")
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    rc = load().hexconv_bwd(
        _dev(x, "x", dt), _dev(dy, "dy", dt, (N, Co, Ho, Wo)),
        _dev(w, "w", dt, (Co, Ci, T)), _dev(dx, "dx", dt, (N, Ci, H, W)),
        _dev(dw, "dw", None, (Co, Ci, T)), _dev(db, "db", None, (Co,)),
        ws_ptr, ws_bytes, N, Ci, Co, H, W, k, stride, dt, _stream(stream))
    _ok("hexconv_bwd", rc)
    return dx, dw, db


HEX_NOALLOC_SCRATCH_BYTES = 64 << 20


def hexconv_bwd_noalloc(x, dy, w, dx, dw, db, k: int, stride: int = 1, stream=None):
    """hexconv_bwd without a workspace: the library's static scratch array
    serves instead (no allocation in the call; overlapping calls on one GPU
    race)."""
    torch = _torch()
    N, Ci, H, W = x.shape
    Co = dw.shape[0]
    dt = _dtype_code(x)
    T = hex_num_taps(k)
    Ho, Wo = hex_out_shape(H, W, k, stride)
    if dw.dtype != torch.float32 or (db is not None and db.dtype != torch.float32):
        raise TypeError("hexconv: dw and db must be float32")
    rc = load().hexconv_bwd_noalloc(
        _dev(x, "x", dt), _dev(dy, "dy", dt, (N, Co, Ho, Wo)),
        _dev(w, "w", dt, (Co, Ci, T)), _dev(dx, "dx", dt, (N, Ci, H, W)),
        _dev(dw, "dw", None, (Co, Ci, T)), _dev(db, "db", None, (Co,)),
        N, Ci, Co, H, W, k, stride, dt, _stream(stream))
    _ok("hexconv_bwd_noalloc", rc)
    return dx, dw, db


def hexpool_fwd(x, y, argmax_tap, k: int, stride: int, mode: int,
                stream=None):
    """y <- hexagonal max (mode 0) or average (mode 1) pooling of x."""
    torch = _torch()
    N, C, H, W = x.shape
    dt = _dtype_code(x)
    Ho, Wo = hex_out_shape(H, W, k, stride)
    if argmax_tap is not None and argmax_tap.dtype != torch.uint8:
        raise TypeError("hexconv: argmax_tap must be uint8")
    rc = load().hexpool_fwd(
        _dev(x, "x", dt), _dev(y, "y", dt, (N, C, Ho, Wo)),
        _dev(argmax_tap, "argmax_tap", None, (N, C, Ho, Wo)),
        N, C, H, W, k, stride, mode, dt, _stream(stream))
    _ok("hexpool_fwd", rc)
    return y


def hexpool_bwd(dy, argmax_tap, relu_y, dx, k: int, stride: int, mode: int,
                stream=None):
    """dx <- pooling gradient (optionally masked by relu_y > 0)."""
    torch = _torch()
    N, C, H, W = dx.shape
    dt = _dtype_code(dx)
    Ho, Wo = hex_out_shape(H, W, k, stride)
    if argmax_tap is not None and argmax_tap.dtype != torch.uint8:
        raise TypeError("hexconv: argmax_tap must be uint8")
    rc = load().hexpool_bwd(
        _dev(dy, "dy", dt, (N, C, Ho, Wo)),
        _dev(argmax_tap, "argmax_tap", None, (N, C, Ho, Wo)),
        _dev(relu_y, "relu_y", dt, (N, C, H, W)), _dev(dx, "dx", dt),
        N, C, H, W, k, stride, mode, dt, _stream(stream))
    _ok("hexpool_bwd", rc)
    return dx


# ------------------------------------------------------- three dimensions
# x[N][C][D][H][W]; window of size (k, kz): the size-k hexagon times the
# planes dz = -kz .. kz; w[C_out][C_in][2kz+1][T]; plane stride stride_z.

def hex_out_shape3d(D: int, H: int, W: int, k: int, kz: int, stride: int, stride_z: int):
    do, ho, wo = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _ok("hex_out_shape3d", load().hex_out_shape3d(D, H, W, k, kz, stride, stride_z,
                                                  ctypes.byref(do), ctypes.byref(ho),
                                                  ctypes.byref(wo)))
    return do.value, ho.value, wo.value


def hexconv3d_fwd(x, w, bias, y, k: int, kz: int, stride: int = 1, stride_z: int = 1,
                  relu: bool = False, stream=None):
    """y <- 3-D hexagonal convolution of x with w (+ bias) (Sec. 2.4)."""
    N, Ci, D, H, W = x.shape
    Co = w.shape[0]
    dt = _dtype_code(x)
    T = hex_num_taps(k)
    Do, Ho, Wo = hex_out_shape3d(D, H, W, k, kz, stride, stride_z)
    rc = load().hexconv3d_fwd(
        _dev(x, "x", dt), _dev(w, "w", dt, (Co, Ci, 2 * kz + 1, T)),
        _dev(bias, "bias", dt, (Co,)), _dev(y, "y", dt, (N, Co, Do, Ho, Wo)),
        N, Ci, Co, D, H, W, k, kz, stride, stride_z, dt, HEX_FLAG_RELU if relu else 0,
        _stream(stream))
    _ok("hexconv3d_fwd", rc)
    return y


def hexconv3d_bwd_data(dy, w, dx, k: int, kz: int, stride: int = 1, stride_z: int = 1,
                       stream=None):
    N, Ci, D, H, W = dx.shape
    Co = w.shape[0]
    dt = _dtype_code(dx)
    T = hex_num_taps(k)
    Do, Ho, Wo = hex_out_shape3d(D, H, W, k, kz, stride, stride_z)
    rc = load().hexconv3d_bwd_data(
        _dev(dy, "dy", dt, (N, Co, Do, Ho, Wo)), _dev(w, "w", dt, (Co, Ci, 2 * kz + 1, T)),
        _dev(dx, "dx", dt), N, Ci, Co, D, H, W, k, kz, stride, stride_z, dt, _stream(stream))
    _ok("hexconv3d_bwd_data", rc)
    return dx


def hexconv3d_bwd_weight_workspace(N, C_in, C_out, D, H, W, k, kz, stride, stride_z, dt):
    return load().hexconv3d_bwd_weight_workspace(N, C_in, C_out, D, H, W, k, kz, stride,
                                                 stride_z, dt)


def hexconv3d_bwd_weight(x, dy, dw, db, ws, k: int, kz: int, stride: int = 1,
                         stride_z: int = 1, stream=None):
    torch = _torch()
    N, Ci, D, H, W = x.shape
    Co = dw.shape[0]
    dt = _dtype_code(x)
    T = hex_num_taps(k)
    Do, Ho, Wo = hex_out_shape3d(D, H, W, k, kz, stride, stride_z)
    if dw.dtype != torch.float32 or (db is not None and db.dtype != torch.float32):
        raise TypeError("hexconv: dw and db must be float32")
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    rc = load().hexconv3d_bwd_weight(
        _dev(x, "x", dt), _dev(dy, "dy", dt, (N, Co, Do, Ho, Wo)),
        _dev(dw, "dw", None, (Co, Ci, 2 * kz + 1, T)), _dev(db, "db", None, (Co,)),
        _dev(ws, "ws"), ws_bytes, N, Ci, Co, D, H, W, k, kz, stride, stride_z, dt,
        _stream(stream))
    _ok("hexconv3d_bwd_weight", rc)
    return dw, db


def hexpool3d_fwd(x, y, argmax, k: int, kz: int, stride: int, stride_z: int, mode: int,
                  stream=None):
    """y <- 3-D max (mode 0) or average (mode 1) pooling; argmax: int16
    tensor (the uint16 tap indices, bit for bit) or None."""
    torch = _torch()
    N, C, D, H, W = x.shape
    dt = _dtype_code(x)
    Do, Ho, Wo = hex_out_shape3d(D, H, W, k, kz, stride, stride_z)
    if argmax is not None and argmax.dtype not in (torch.int16, torch.uint16):
        raise TypeError("hexconv: 3-D argmax must be a 16-bit tensor")
    rc = load().hexpool3d_fwd(
        _dev(x, "x", dt), _dev(y, "y", dt, (N, C, Do, Ho, Wo)),
        _dev(argmax, "argmax", None, (N, C, Do, Ho, Wo)),
        N, C, D, H, W, k, kz, stride, stride_z, mode, dt, _stream(stream))
    _ok("hexpool3d_fwd", rc)
    return y


def hexpool3d_bwd(dy, argmax, relu_y, dx, k: int, kz: int, stride: int, stride_z: int,
                  mode: int, stream=None):
    torch = _torch()
    N, C, D, H, W = dx.shape
    dt = _dtype_code(dx)
    Do, Ho, Wo = hex_out_shape3d(D, H, W, k, kz, stride, stride_z)
    if argmax is not None and argmax.dtype not in (torch.int16, torch.uint16):
        raise TypeError("hexconv: 3-D argmax must be a 16-bit tensor")
    rc = load().hexpool3d_bwd(
        _dev(dy, "dy", dt, (N, C, Do, Ho, Wo)),
        _dev(argmax, "argmax", None, (N, C, Do, Ho, Wo)),
        _dev(relu_y, "relu_y", dt, (N, C, D, H, W)), _dev(dx, "dx", dt),
        N, C, D, H, W, k, kz, stride, stride_z, mode, dt, _stream(stream))
    _ok("hexpool3d_bwd", rc)
    return dx
