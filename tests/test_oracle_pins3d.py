"""Pins for the fp64 reference's three-dimensional operations (hexagonal x-y
planes, equidistant samples along z; HexagDLy, arXiv:1903.01814, Sec. 2.4
"Software Functionalities"), checked against facts other than the oracle
itself: the independent physical-position brute force (oracle/brute.py),
the 2-D operations it must reduce to (themselves pinned in
test_oracle_pins.py), delta responses, the z-reflection symmetry, adjoint
identities and pooling identities.  A plausible slip -- a flipped dz, a
dropped plane, the z stride applied to the wrong axis, the wrong weight
index order, a wrong plane count -- fails at least one of them.
"""
import numpy as np
import pytest

import oracle
from oracle import brute


def _rng(seed):
    return np.random.default_rng(seed)


@pytest.mark.parametrize("sz", [1, 2, 3, 5])
def test_out_shape3d(sz):
    """Centres on the planes 0, sz, 2sz, ... below D: ceil(D / sz) planes;
    the hexagonal plane follows the 2-D rule."""
    for D in range(1, 14):
        for (H, W, s) in [(5, 5, 2), (9, 8, 1), (12, 13, 3)]:
            Do, Ho, Wo = oracle.out_shape3d(D, H, W, s, sz)
            assert Do == -(-D // sz) == len(brute.z_centres(D, sz))
            assert (Ho, Wo) == oracle.out_shape(H, W, s)


CASES = [
    # N, Ci, Co, D, H, W, k, kz, s, sz
    (1, 1, 1, 4, 5, 6, 1, 1, 1, 1), (2, 2, 3, 5, 6, 5, 1, 1, 1, 2),
    (1, 2, 2, 3, 7, 7, 2, 1, 2, 1), (1, 1, 2, 6, 5, 7, 0, 2, 1, 3),
    (1, 2, 1, 1, 6, 6, 1, 2, 1, 1), (1, 1, 1, 7, 8, 9, 2, 0, 3, 2),
    (2, 1, 2, 5, 4, 5, 1, 3, 2, 2),
]


@pytest.mark.parametrize("case", CASES)
def test_conv3d_matches_physical_brute_force(case):
    """The oracle's axial algebra against the brute force that places every
    element physically (planes at equidistant heights)."""
    N, Ci, Co, D, H, W, k, kz, s, sz = case
    rng = _rng(sum(case))
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, D, H, W))
    w = rng.normal(size=(Co, Ci, 2 * kz + 1, T))
    b = rng.normal(size=Co)
    np.testing.assert_allclose(oracle.conv3d_fwd(x, w, b, k, kz, s, sz),
                               brute.conv3d_fwd(x, w, b, k, kz, s, sz), rtol=0, atol=1e-12)


@pytest.mark.parametrize("k,kz", [(1, 1), (2, 1), (1, 2)])
def test_conv3d_delta_response(k, kz):
    """A delta at an interior element (z0, r0, c0) is read by the window of
    every centre it lies in: the output at plane z0 - dz, element (r0, c0)
    moved by minus tap t, equals w[dz][t]; all other outputs are zero, so
    exactly (2kz+1) * T outputs are non-zero."""
    D, H, W = 2 * kz + 5, 4 * k + 6, 4 * k + 7
    z0, r0, c0 = kz + 2, 2 * k + 2, 2 * k + 3
    T = oracle.num_taps(k)
    x = np.zeros((1, 1, D, H, W))
    x[0, 0, z0, r0, c0] = 1.0
    w = np.arange(1, (2 * kz + 1) * T + 1, dtype=np.float64).reshape(1, 1, 2 * kz + 1, T)
    y = oracle.conv3d_fwd(x, w, None, k, kz)
    dq, ds = oracle.taps(k)
    want = np.zeros_like(y)
    for h in range(-kz, kz + 1):
        for t in range(T):
            r, c = oracle.step(r0, c0, -int(dq[t]), -int(ds[t]))
            want[0, 0, z0 - h, r, c] = w[0, 0, h + kz, t]
    np.testing.assert_array_equal(y, want)
    assert np.count_nonzero(y) == (2 * kz + 1) * T


@pytest.mark.parametrize("sz", [1, 2])
def test_conv3d_depth_one_kernel_is_2d(sz):
    """kz = 0: every output plane is the 2-D convolution of its centre input
    plane (planes sz*l)."""
    rng = _rng(3)
    N, Ci, Co, D, H, W, k, s = 2, 2, 3, 7, 9, 8, 2, 2
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, D, H, W))
    w = rng.normal(size=(Co, Ci, 1, T))
    b = rng.normal(size=Co)
    y = oracle.conv3d_fwd(x, w, b, k, 0, s, sz)
    for l in range(y.shape[2]):
        np.testing.assert_allclose(y[:, :, l], oracle.conv_fwd(x[:, :, sz * l], w[:, :, 0], b, k, s),
                                   rtol=0, atol=1e-12)


def test_conv3d_single_plane_uses_centre_weights():
    """D = 1 with kz > 0: the planes above and below are padding, so only
    the centre plane's weights act (2-D convolution with w[:, :, kz])."""
    rng = _rng(4)
    k, kz = 1, 2
    T = oracle.num_taps(k)
    x = rng.normal(size=(2, 3, 1, 8, 9))
    w = rng.normal(size=(4, 3, 2 * kz + 1, T))
    y = oracle.conv3d_fwd(x, w, None, k, kz)
    np.testing.assert_allclose(y[:, :, 0], oracle.conv_fwd(x[:, :, 0], w[:, :, kz], None, k, 1),
                               rtol=0, atol=1e-12)


def test_conv3d_z_reflection():
    """Reversing the planes of the input and of the kernel reverses the
    output planes (stride 1 along z): the window is symmetric in z."""
    rng = _rng(5)
    k, kz = 1, 2
    T = oracle.num_taps(k)
    x = rng.normal(size=(1, 2, 6, 7, 8))
    w = rng.normal(size=(2, 2, 2 * kz + 1, T))
    y = oracle.conv3d_fwd(x, w, None, k, kz)
    yf = oracle.conv3d_fwd(x[:, :, ::-1], w[:, :, ::-1], None, k, kz)
    np.testing.assert_allclose(yf, y[:, :, ::-1], rtol=0, atol=1e-12)


@pytest.mark.parametrize("s,sz", [(1, 1), (2, 1), (1, 2), (2, 3), (3, 2)])
def test_conv3d_adjoint_identities(s, sz):
    """<fwd(x), dy> = <x, bwd_data(dy)> (no bias); <dw, V> = <fwd_V(x), dy>
    for any kernel V; db = sum of dy."""
    rng = _rng(10 * s + sz)
    N, Ci, Co, D, H, W, k, kz = 2, 3, 2, 7, 9, 10, 1, 1
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, D, H, W))
    w = rng.normal(size=(Co, Ci, 2 * kz + 1, T))
    y = oracle.conv3d_fwd(x, w, None, k, kz, s, sz)
    dy = rng.normal(size=y.shape)
    dx = oracle.conv3d_bwd_data(dy, w, k, kz, s, sz, D, H, W)
    assert abs(np.vdot(y, dy) - np.vdot(x, dx)) <= 1e-10 * np.abs(y).sum()
    dw, db = oracle.conv3d_bwd_weight(x, dy, k, kz, s, sz)
    V = rng.normal(size=w.shape)
    lhs = np.vdot(dw, V)
    rhs = np.vdot(oracle.conv3d_fwd(x, V, None, k, kz, s, sz), dy)
    assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(rhs))
    np.testing.assert_allclose(db, dy.sum(axis=(0, 2, 3, 4)), rtol=1e-13, atol=1e-12)


@pytest.mark.parametrize("mode", [oracle.POOL_MAX, oracle.POOL_AVG])
@pytest.mark.parametrize("case", [(1, 2, 4, 5, 6, 1, 1, 1, 1), (2, 1, 5, 7, 6, 1, 1, 2, 2),
                                  (1, 2, 3, 6, 7, 2, 0, 1, 2), (1, 1, 6, 5, 5, 0, 2, 1, 3)])
def test_pool3d_matches_physical_brute_force(case, mode):
    """Max and average pooling, and the max's first maximal tap, against the
    physical brute force; plateaus make ties."""
    N, C, D, H, W, k, kz, s, sz = case
    rng = _rng(sum(case) + mode)
    x = rng.normal(size=(N, C, D, H, W))
    x[0, 0, :2, :3, :3] = 0.75
    y, am = oracle.pool3d_fwd(x, k, kz, s, sz, mode)
    yb, amb = brute.pool3d_fwd(x, k, kz, s, sz, mode)
    np.testing.assert_allclose(y, yb, rtol=0, atol=1e-12)
    if mode == oracle.POOL_MAX:
        np.testing.assert_array_equal(am, amb)


def test_pool3d_depth_one_window_is_2d():
    """kz = 0: 3-D pooling is the 2-D pooling of the centre planes,
    argmax included."""
    rng = _rng(8)
    x = rng.normal(size=(2, 3, 6, 9, 8))
    for mode in (oracle.POOL_MAX, oracle.POOL_AVG):
        y, am = oracle.pool3d_fwd(x, 1, 0, 2, 2, mode)
        for l in range(y.shape[2]):
            y2, am2 = oracle.pool_fwd(x[:, :, 2 * l], 1, 2, mode)
            np.testing.assert_array_equal(y[:, :, l], y2)
            if mode == oracle.POOL_MAX:
                np.testing.assert_array_equal(am[:, :, l], am2)


def test_pool3d_tie_across_planes_keeps_lowest_plane():
    """Equal maxima in the planes below and above the centre: the first in
    tap order (planes ascending) wins."""
    k, kz = 1, 1
    T = oracle.num_taps(k)
    x = np.full((1, 1, 3, 5, 5), -1.0)
    x[0, 0, 0, 2, 2] = 3.0
    x[0, 0, 2, 2, 2] = 3.0
    y, am = oracle.pool3d_fwd(x, k, kz, 1, 1, oracle.POOL_MAX)
    assert y[0, 0, 1, 2, 2] == 3.0
    assert am[0, 0, 1, 2, 2] == 0 * T + T // 2        # plane dz = -1, centre tap


def test_pool3d_average_of_constant():
    """Average of a constant c: c where the whole window is inside, else c
    times the fraction of in-tensor taps ((2kz+1) T in the divisor)."""
    k, kz = 1, 1
    T = oracle.num_taps(k)
    x = np.full((1, 1, 5, 8, 8), 2.0)
    y, _ = oracle.pool3d_fwd(x, k, kz, 1, 1, oracle.POOL_AVG)
    assert y[0, 0, 2, 4, 4] == pytest.approx(2.0)
    # plane 0: the plane below is padding, the hexagon is inside
    assert y[0, 0, 0, 4, 4] == pytest.approx(2.0 * 2 * T / (3 * T))


@pytest.mark.parametrize("s,sz", [(1, 1), (2, 2), (1, 3)])
def test_pool3d_backward(s, sz):
    """Average: the gradient is the adjoint of the (linear) forward.  Max:
    with positive inputs padding never wins, and routing dy to the argmax
    element gives <dx, x> = <dy, y>.  A ReLU mask zeroes the masked
    elements."""
    rng = _rng(20 + s + sz)
    k, kz = 1, 1
    N, C, D, H, W = 2, 2, 6, 7, 8
    x = rng.uniform(0.1, 1.0, size=(N, C, D, H, W))
    ya, _ = oracle.pool3d_fwd(x, k, kz, s, sz, oracle.POOL_AVG)
    dy = rng.normal(size=ya.shape)
    dxa = oracle.pool3d_bwd(dy, None, None, k, kz, s, sz, oracle.POOL_AVG, D, H, W)
    assert abs(np.vdot(ya, dy) - np.vdot(x, dxa)) <= 1e-12 * np.abs(ya).sum()
    ym, am = oracle.pool3d_fwd(x, k, kz, s, sz, oracle.POOL_MAX)
    dxm = oracle.pool3d_bwd(dy, am, None, k, kz, s, sz, oracle.POOL_MAX, D, H, W)
    assert abs(np.vdot(ym, dy) - np.vdot(x, dxm)) <= 1e-12 * np.abs(ym).sum()
    relu_y = rng.normal(size=x.shape)
    dxr = oracle.pool3d_bwd(dy, am, relu_y, k, kz, s, sz, oracle.POOL_MAX, D, H, W)
    np.testing.assert_array_equal(dxr, np.where(relu_y > 0, dxm, 0.0))
