"""CPU checks of the generic kernels' launch plans (csrc/generic_plan.h,
compiled here with g++): for every kernel size and stride the ABI accepts,
and every channel regime, the forward and data-gradient plans fit the LDS a
block may use (input region plus staged weights), tiles fit the block, and
a budget too small for any tile is reported as not fitting (the ABI then
returns HEX_ERR_UNSUPPORTED before enqueuing anything)."""
import ctypes
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1903_01814_amd", "csrc")
SRC = os.path.join(ROOT, "tests", "native", "plan_query.cpp")

CHANNELS = [1, 2, 7, 8, 9, 31, 32, 33, 63, 64, 65, 128, 512]


@pytest.fixture(scope="module")
def lib(tmp_path_factory):
    so = str(tmp_path_factory.mktemp("plan") / "libplan.so")
    subprocess.run(["g++", "-std=c++17", "-O1", "-shared", "-fPIC", "-Wall", "-Werror",
                    "-I", CSRC, SRC, "-o", so], check=True)
    lib = ctypes.CDLL(so)
    L = ctypes.c_long
    lib.plan_fwd_query.argtypes = [ctypes.c_int] * 4 + [L, ctypes.POINTER(L)]
    lib.plan_bwd_data_query.argtypes = [ctypes.c_int] * 3 + [L, ctypes.POINTER(L)]
    lib.plan_lds_limit.restype = L
    return lib


def fwd(lib, ci, co, k, s, limit):
    out = (ctypes.c_long * 6)()
    lib.plan_fwd_query(ci, co, k, s, limit, out)
    return list(out)


def bwd(lib, ci, co, k, limit):
    out = (ctypes.c_long * 4)()
    lib.plan_bwd_data_query(ci, co, k, limit, out)
    return list(out)


def taps(k):
    return 1 + 3 * k * (k + 1)


def region_floats(TI, TJ, k, s):
    rows = s * (TI - 1) + s // 2 + 2 * k + 1
    cols = s * (TJ - 1) + 2 * k + 1
    return (rows * cols + 3) & ~3


@pytest.mark.parametrize("k", range(0, 9))
@pytest.mark.parametrize("s", range(1, 9))
def test_forward_plan_fits(lib, k, s):
    limit = lib.plan_lds_limit()
    assert limit == 64 * 1024
    for ci in CHANNELS:
        for co in CHANNELS:
            ok, TI, TJ, cb, G, lds = fwd(lib, ci, co, k, s, limit)
            assert ok, (ci, co, k, s)
            assert 1 <= TI * TJ <= 256
            assert cb in (8, 32, 64) and (cb == 8 or co >= cb)
            assert 1 <= G <= min(8, ci)
            # the LDS the kernel indexes: G regions and G x T x cb weights
            need = 4 * G * (region_floats(TI, TJ, k, s) + taps(k) * cb)
            assert lds == need <= limit, (ci, co, k, s, lds)


@pytest.mark.parametrize("k", range(0, 9))
def test_data_gradient_plan_fits(lib, k):
    limit = lib.plan_lds_limit()
    for ci in CHANNELS:
        for co in CHANNELS:
            ok, cb, CC, lds = bwd(lib, ci, co, k, limit)
            assert ok and cb in (8, 32, 64) and 1 <= CC <= co
            assert lds == 4 * CC * taps(k) * cb <= limit, (ci, co, k, lds)


def test_largest_kernel_and_stride_regression(lib):
    """k = 8, stride 8, 64 output channels: the region alone fitted the old
    budget while region plus weights (about 95 KB) did not; the plan now
    keeps both within it by staging fewer output channels per block."""
    limit = lib.plan_lds_limit()
    ok, TI, TJ, cb, G, lds = fwd(lib, 64, 64, 8, 8, limit)
    assert ok and lds <= limit and cb == 32


def test_plan_reports_no_fit(lib):
    """A budget below any tile's needs is reported as not fitting (the ABI's
    HEX_ERR_UNSUPPORTED path)."""
    assert fwd(lib, 1, 1, 8, 8, 4096)[0] == 0
    assert bwd(lib, 64, 64, 8, 4096)[0] == 0
    assert fwd(lib, 1, 1, 1, 1, 4096)[0] == 1
