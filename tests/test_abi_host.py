"""Host-side checks of libhexconv (no GPU needed): every symbol the public
header declares is exported, the library's geometry tables agree bit for bit
with the oracle's independent enumeration, and every argument error is
rejected on the host before anything is enqueued."""
import ctypes
import os
import re

import pytest

import oracle
from paper_1903_01814_amd import hexconv as hx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hexconv.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(hex\w+)\s*\(", src,
                                 flags=re.M)))


def test_header_declares_expected_entry_points():
    names = declared_functions()
    for n in ["hexconv_fwd", "hexconv_bwd_data", "hexconv_bwd_weight",
              "hexconv_bwd_weight_workspace", "hexpool_fwd", "hexpool_bwd",
              "hexconv_bwd", "hexconv_bwd_workspace", "hexconv_bwd_noalloc",
              "hex_num_taps", "hex_out_shape", "hex_tap_table",
              "hex_status_string"]:
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = hx.load()
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert name in hx.SIGNATURES, name


@pytest.mark.parametrize("k", range(0, 9))
@pytest.mark.parametrize("parity", [0, 1])
def test_tap_table_matches_oracle(k, parity):
    """Library tap tables vs the oracle's axial enumeration, bit-exact."""
    assert hx.hex_num_taps(k) == oracle.num_taps(k)
    dcol, drow = hx.hex_tap_table(k, parity)
    dq, ds = oracle.taps(k)
    r0, c0 = 20, 20 + parity
    for t in range(len(dq)):
        r, c = oracle.step(r0, c0, int(dq[t]), int(ds[t]))
        assert (dcol[t], drow[t]) == (c - c0, r - r0)


def test_out_shape_matches_oracle():
    # the output lattice does not depend on the kernel size (centres sit on
    # tensor elements, Sec. 2.3): every k gives the same shape
    for s in range(1, 9):
        for H in list(range(1, 20)) + [40, 48, 128, 257]:
            for W in list(range(1, 14)) + [40, 48, 128, 255]:
                want = oracle.out_shape(H, W, s)
                for k in (0, 1, 5, 8):
                    assert hx.hex_out_shape(H, W, k, s) == want, (H, W, k, s)


def test_status_strings():
    for st in (0, -1, -2, -3):
        assert hx.status_string(st).startswith("HEX_")
    assert "unknown" in hx.status_string(7)


# ----------------------------------------------------------- error paths

class FakePtr:
    """Aligned, never-dereferenced addresses: validation must reject bad
    arguments before touching memory or the GPU."""
    A = 0x10000
    B = 0x20000
    C = 0x30000
    D = 0x40000
    E = 0x50000
    F = 0x60000


def _fwd(x=FakePtr.A, w=FakePtr.B, b=None, y=FakePtr.C, N=2, Ci=1, Co=4, H=8,
         W=8, k=1, s=1, dt=0, flags=0):
    return hx.load().hexconv_fwd(x, w, b, y, N, Ci, Co, H, W, k, s, dt, flags,
                                 None)


@pytest.mark.parametrize("kw", [
    dict(x=None), dict(w=None), dict(y=None), dict(x=FakePtr.A + 4),
    dict(b=FakePtr.D + 2), dict(N=-1), dict(Ci=0), dict(Co=0), dict(H=0),
    dict(W=0), dict(k=-1), dict(k=9), dict(s=0), dict(s=9), dict(dt=2),
    dict(dt=-1), dict(flags=2)])
def test_fwd_rejects_invalid(kw):
    assert _fwd(**kw) == hx.HEX_ERR_INVALID_ARG


def test_fwd_rejects_oversize():
    assert _fwd(N=1 << 20, Ci=64, H=256, W=256) == hx.HEX_ERR_UNSUPPORTED
    assert _fwd(H=70000) == hx.HEX_ERR_UNSUPPORTED


def test_fwd_empty_batch_is_noop():
    # N == 0 or an empty output: nothing to compute, nothing enqueued; an
    # empty batch may come with NULL buffers (empty tensors)
    assert _fwd(N=0) == hx.HEX_OK
    assert _fwd(N=0, x=None, y=None, w=None) == hx.HEX_OK
    assert _fwd(H=1, W=5, s=2) == hx.HEX_OK
    lib = hx.load()
    assert lib.hexconv_bwd_data(None, None, None, 0, 1, 2, 8, 8, 1, 1, 0, None) == hx.HEX_OK
    assert lib.hexpool_fwd(None, None, None, 0, 3, 8, 8, 1, 2, 0, 1, None) == hx.HEX_OK
    assert lib.hexpool_bwd(None, None, None, None, 0, 3, 8, 8, 1, 2, 0, 1, None) == hx.HEX_OK
    # the weight gradient of an empty batch is zero, so dw is still required
    assert lib.hexconv_bwd_weight(None, None, None, None, None, 0, 0, 1, 2, 8, 8, 1,
                                  1, 0, None) == hx.HEX_ERR_INVALID_ARG


def test_bwd_data_rejects_invalid():
    lib = hx.load()
    f = lambda dy=FakePtr.A, w=FakePtr.B, dx=FakePtr.C, k=1, s=1, dt=0: \
        lib.hexconv_bwd_data(dy, w, dx, 2, 3, 4, 9, 9, k, s, dt, None)
    assert f(dy=None) == hx.HEX_ERR_INVALID_ARG
    assert f(w=None) == hx.HEX_ERR_INVALID_ARG
    assert f(dx=None) == hx.HEX_ERR_INVALID_ARG
    assert f(dx=FakePtr.C + 8) == hx.HEX_ERR_INVALID_ARG
    assert f(k=12) == hx.HEX_ERR_INVALID_ARG
    assert f(dt=5) == hx.HEX_ERR_INVALID_ARG


def test_bwd_weight_workspace_and_errors():
    lib = hx.load()
    need = lib.hexconv_bwd_weight_workspace(4, 2, 3, 16, 16, 1, 1, 0)
    assert need > 0
    assert lib.hexconv_bwd_weight_workspace(4, 2, 3, 16, 16, -1, 1, 0) == 0
    f = lambda x=FakePtr.A, dy=FakePtr.B, dw=FakePtr.C, db=None, ws=FakePtr.D, \
        nb=need: lib.hexconv_bwd_weight(x, dy, dw, db, ws, nb, 4, 2, 3, 16, 16,
                                        1, 1, 0, None)
    assert f(ws=None) == hx.HEX_ERR_INVALID_ARG
    assert f(nb=need - 1) == hx.HEX_ERR_INVALID_ARG
    assert f(dw=None) == hx.HEX_ERR_INVALID_ARG
    assert f(x=None) == hx.HEX_ERR_INVALID_ARG
    assert f(db=FakePtr.C + 4) == hx.HEX_ERR_INVALID_ARG


def test_bwd_combined_workspace_and_errors():
    """hexconv_bwd: every argument is checked before anything is enqueued,
    for the fused float32 path (1 -> 16 channels, k = 2) and for the
    fallback that runs the two gradients one after the other."""
    lib = hx.load()
    for (Ci, Co, k, dt) in [(1, 16, 2, 0), (3, 5, 1, 1)]:
        need = lib.hexconv_bwd_workspace(4, Ci, Co, 16, 16, k, 1, dt)
        assert need > 0
        assert lib.hexconv_bwd_workspace(4, Ci, Co, 16, 16, -1, 1, dt) == 0
        f = lambda x=FakePtr.A, dy=FakePtr.B, w=FakePtr.C, dx=FakePtr.D, \
            dw=FakePtr.E, db=None, ws=FakePtr.F, nb=need: lib.hexconv_bwd(
                x, dy, w, dx, dw, db, ws, nb, 4, Ci, Co, 16, 16, k, 1, dt, None)
        assert f(ws=None) == hx.HEX_ERR_INVALID_ARG
        assert f(nb=need - 1) == hx.HEX_ERR_INVALID_ARG
        assert f(dw=None) == hx.HEX_ERR_INVALID_ARG
        assert f(x=None) == hx.HEX_ERR_INVALID_ARG
        assert f(dy=None) == hx.HEX_ERR_INVALID_ARG
        assert f(w=None) == hx.HEX_ERR_INVALID_ARG        # dx wanted, no weights
        assert f(dx=FakePtr.D + 4) == hx.HEX_ERR_INVALID_ARG
        assert f(db=FakePtr.C + 4) == hx.HEX_ERR_INVALID_ARG
        assert lib.hexconv_bwd(FakePtr.A, FakePtr.B, FakePtr.C, FakePtr.D, FakePtr.E,
                               None, FakePtr.F, need, 4, Ci, Co, 16, 16, 9, 1, dt,
                               None) == hx.HEX_ERR_INVALID_ARG


def test_pool_rejects_invalid():
    lib = hx.load()
    fw = lambda x=FakePtr.A, y=FakePtr.B, am=None, mode=0, k=1, s=2: \
        lib.hexpool_fwd(x, y, am, 2, 3, 9, 9, k, s, mode, 1, None)
    assert fw(x=None) == hx.HEX_ERR_INVALID_ARG
    assert fw(mode=2) == hx.HEX_ERR_INVALID_ARG
    assert fw(am=FakePtr.C + 1) == hx.HEX_ERR_INVALID_ARG
    assert fw(s=0) == hx.HEX_ERR_INVALID_ARG
    bw = lambda dy=FakePtr.A, am=FakePtr.B, ry=None, dx=FakePtr.C, mode=0: \
        lib.hexpool_bwd(dy, am, ry, dx, 2, 3, 9, 9, 1, 2, mode, 1, None)
    assert bw(am=None) == hx.HEX_ERR_INVALID_ARG          # max needs argmax
    assert bw(dx=None) == hx.HEX_ERR_INVALID_ARG
    assert bw(ry=FakePtr.D + 2) == hx.HEX_ERR_INVALID_ARG
    assert bw(mode=3) == hx.HEX_ERR_INVALID_ARG


def test_noalloc_rejects_oversized_workspace():
    """hexconv_bwd_noalloc: a shape whose workspace exceeds the static
    scratch array is HEX_ERR_UNSUPPORTED, decided on the host before any
    HIP call (fake pointers are never touched); bad arguments are rejected
    like hexconv_bwd's."""
    lib = hx.load()
    big = (64, 512, 256, 128, 128, 8, 1, hx.HEX_F32)
    assert hx.hexconv_bwd_workspace(*big) > hx.HEX_NOALLOC_SCRATCH_BYTES
    A, B, C, D, E, F = (FakePtr.A, FakePtr.B, FakePtr.C, FakePtr.D, FakePtr.E, FakePtr.F)
    assert lib.hexconv_bwd_noalloc(A, B, C, D, E, F, *big, None) == hx.HEX_ERR_UNSUPPORTED
    ok = (2, 1, 4, 16, 16, 1, 1, hx.HEX_F32)
    assert lib.hexconv_bwd_noalloc(A, B, C, D, None, F, *ok, None) == hx.HEX_ERR_INVALID_ARG
    assert lib.hexconv_bwd_noalloc(A, B, None, D, E, F, *ok, None) == hx.HEX_ERR_INVALID_ARG
    assert lib.hexconv_bwd_noalloc(A, B, C, D + 4, E, F, *ok, None) == hx.HEX_ERR_INVALID_ARG
    assert lib.hexconv_bwd_noalloc(A, B, C, D, E, F, 2, 1, 4, 16, 16, 9, 1, 0,
                                   None) == hx.HEX_ERR_INVALID_ARG


def test_host_helper_errors():
    lib = hx.load()
    assert lib.hex_num_taps(-1) == hx.HEX_ERR_INVALID_ARG
    assert lib.hex_num_taps(9) == hx.HEX_ERR_INVALID_ARG
    a, b = ctypes.c_int(), ctypes.c_int()
    assert lib.hex_out_shape(0, 5, 1, 1, ctypes.byref(a), ctypes.byref(b)) == -1
    assert lib.hex_out_shape(5, 5, 1, 1, None, ctypes.byref(b)) == -1
    assert lib.hex_out_shape(5, 5, -1, 1, ctypes.byref(a), ctypes.byref(b)) == -1
    assert lib.hex_out_shape(5, 5, 9, 1, ctypes.byref(a), ctypes.byref(b)) == -1
    assert lib.hex_out_shape(5, 5, 1, 0, ctypes.byref(a), ctypes.byref(b)) == -1
    buf = (ctypes.c_int * 7)()
    assert lib.hex_tap_table(1, 2, buf, buf) == -1
    assert lib.hex_tap_table(1, 0, None, buf) == -1


def test_timing_host_paths():
    """Kernel timing with nothing launched reports nothing; bad output
    arguments are rejected."""
    hx.hexconv_timing_begin()
    assert hx.hexconv_timing_end() == {}
    lib = hx.load()
    n = ctypes.c_int()
    counts = (ctypes.c_int * 1)()
    total = (ctypes.c_double * 1)()
    names = ctypes.create_string_buffer(hx.HEX_TIMING_NAME_LEN)
    assert lib.hexconv_timing_end(0, names, counts, total, ctypes.byref(n)) == hx.HEX_ERR_INVALID_ARG
    assert lib.hexconv_timing_end(1, None, counts, total, ctypes.byref(n)) == hx.HEX_ERR_INVALID_ARG


def test_out_shape3d_matches_oracle():
    for sz in range(1, 9):
        for D in range(1, 12):
            for (H, W, s) in [(5, 5, 2), (40, 40, 1), (9, 12, 3), (1, 5, 2)]:
                want = oracle.out_shape3d(D, H, W, s, sz)
                for k, kz in ((0, 0), (1, 4), (8, 2)):
                    assert hx.hex_out_shape3d(D, H, W, k, kz, s, sz) == want


def test_3d_argument_errors():
    """3-D entry points reject bad sizes, window depths, plane strides,
    modes and pointers on the host (fake pointers are never touched)."""
    lib = hx.load()
    A, B, C, D_, E = FakePtr.A, FakePtr.B, FakePtr.C, FakePtr.D, FakePtr.E
    a, b, c = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    shp = lambda D=4, kz=1, sz=1: lib.hex_out_shape3d(D, 8, 8, 1, kz, 1, sz, ctypes.byref(a),
                                                      ctypes.byref(b), ctypes.byref(c))
    assert shp() == 0 and (a.value, b.value, c.value) == (4, 8, 8)
    assert shp(D=0) == hx.HEX_ERR_INVALID_ARG
    assert shp(kz=hx.HEX_MAX_KZ + 1) == hx.HEX_ERR_INVALID_ARG
    assert shp(kz=-1) == hx.HEX_ERR_INVALID_ARG
    assert shp(sz=0) == hx.HEX_ERR_INVALID_ARG
    assert shp(sz=9) == hx.HEX_ERR_INVALID_ARG

    def fwd(x=A, w=B, y=C, N=2, D=4, kz=1, sz=1, flags=0, dt=0):
        return lib.hexconv3d_fwd(x, w, None, y, N, 2, 3, D, 8, 8, 1, kz, 1, sz, dt, flags, None)
    assert fwd(kz=5) == hx.HEX_ERR_INVALID_ARG
    assert fwd(sz=0) == hx.HEX_ERR_INVALID_ARG
    assert fwd(D=0) == hx.HEX_ERR_INVALID_ARG
    assert fwd(x=None) == hx.HEX_ERR_INVALID_ARG
    assert fwd(y=C + 8) == hx.HEX_ERR_INVALID_ARG
    assert fwd(flags=2) == hx.HEX_ERR_INVALID_ARG
    assert fwd(dt=5) == hx.HEX_ERR_INVALID_ARG
    assert fwd(N=0) == hx.HEX_OK                       # empty batch: nothing enqueued
    assert fwd(D=70000) == hx.HEX_ERR_UNSUPPORTED
    assert lib.hexconv3d_bwd_data(A, B, None, 2, 2, 3, 4, 8, 8, 1, 1, 1, 1, 0,
                                  None) == hx.HEX_ERR_INVALID_ARG
    assert lib.hexconv3d_bwd_weight(A, B, C, None, None, 0, 2, 2, 3, 4, 8, 8, 1, 1, 1, 1, 0,
                                    None) == hx.HEX_ERR_INVALID_ARG   # workspace missing
    assert hx.hexconv3d_bwd_weight_workspace(2, 2, 3, 4, 8, 8, 1, 9, 1, 1, 0) == 0
    assert lib.hexpool3d_fwd(A, B, C, 2, 3, 4, 8, 8, 1, 1, 1, 1, 2, 0,
                             None) == hx.HEX_ERR_INVALID_ARG          # mode
    assert lib.hexpool3d_bwd(A, None, None, D_, 2, 3, 4, 8, 8, 1, 1, 1, 1, 0, 0,
                             None) == hx.HEX_ERR_INVALID_ARG          # max needs argmax
