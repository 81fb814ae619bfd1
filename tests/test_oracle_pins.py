"""Pins for the fp64 reference: checks of oracle/ against facts fixed by the
HexagDLy paper (arXiv:1903.01814) and by mathematics, not against itself.

Each test names the passage or property it pins.  A plausible slip in the
oracle (a dropped term, a wrong sign, the wrong parity, a transposed weight
index, a wrong stride lattice) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest

import oracle
from oracle import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SQ = math.sqrt(3.0) / 2.0


def _rng(seed=0):
    return np.random.default_rng(seed)


def _read_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([int(v) for v in line.split()])
    return rows


def _pos(r, c):
    return brute.position(r, c)


# --------------------------------------------------------------- geometry

@pytest.mark.parametrize("k", range(9))
def test_tap_count_closed_form(k):
    """Sec. 2.2: k layers of neighbours around the centre -> 1 + 3k(k+1)."""
    assert oracle.num_taps(k) == 1 + 3 * k * (k + 1)
    if k <= 4:
        assert len(brute.kernel_offsets(k)) == oracle.num_taps(k)


@pytest.mark.parametrize("k", range(1, 7))
def test_column_structure(k):
    """Sec. 2.2 / Fig. 2: the kernel is a set of columns; columns at offset
    +-i hold 2k+1-i contiguous taps, so the +-i pairs form k equal-length
    groups plus the centre column (k+1 sub-kernels)."""
    dq, ds = oracle.taps(k)
    for off in range(-k, k + 1):
        col = ds[dq == off]
        assert len(col) == 2 * k + 1 - abs(off)
        assert np.all(np.diff(col) == 1)          # contiguous, top to bottom
    groups = {len(ds[dq == off]) for off in range(-k, k + 1)}
    assert len(groups) == k + 1


@pytest.mark.parametrize("par", [0, 1])
def test_six_unit_neighbours(par):
    """Sec. 2.1: an interior pixel has exactly six neighbours, all one pitch
    away, for both column parities (checked on physical positions)."""
    r0, c0 = 6, 6 + par
    x0, y0 = _pos(r0, c0)
    dq, ds = oracle.taps(1)
    seen = set()
    for a, b in zip(dq, ds):
        r, c = oracle.step(r0, c0, int(a), int(b))
        d = math.hypot(_pos(r, c)[0] - x0, _pos(r, c)[1] - y0)
        if (a, b) == (0, 0):
            assert (r, c) == (r0, c0)
        else:
            assert abs(d - 1.0) < 1e-12
        seen.add((r, c))
    assert len(seen) == 7
    # no other element within 1.01 pitches
    for r in range(r0 - 3, r0 + 4):
        for c in range(c0 - 3, c0 + 4):
            x, y = _pos(r, c)
            if math.hypot(x - x0, y - y0) < 1.01:
                assert (r, c) in seen


@pytest.mark.parametrize("k", range(0, 5))
@pytest.mark.parametrize("par", [0, 1])
def test_taps_match_neighbour_layers(k, par):
    """Sec. 2.2: tap t of the oracle lands on the same physical displacement
    as the t-th element of the breadth-first neighbour layers (canonical
    order: column by column, top to bottom), for both parities -- so a
    weight belongs to one physical direction."""
    offs = brute.kernel_offsets(k)
    r0, c0 = 10, 10 + par
    x0, y0 = _pos(r0, c0)
    dq, ds = oracle.taps(k)
    for t, (a, b) in enumerate(zip(dq, ds)):
        r, c = oracle.step(r0, c0, int(a), int(b))
        x, y = _pos(r, c)
        assert abs(x - x0 - offs[t][0]) < 1e-9
        assert abs(y - y0 - offs[t][1]) < 1e-9


def test_golden_tap_tables():
    """Hand-derived per-parity tables (tests/golden/taps_k1_k2.txt)."""
    rows = _read_rows("taps_k1_k2.txt")
    for k, par, t, dcol, drow in rows:
        dq, ds = oracle.taps(k)
        r0, c0 = 10, 10 + par
        r, c = oracle.step(r0, c0, int(dq[t]), int(ds[t]))
        assert (c - c0, r - r0) == (dcol, drow), (k, par, t)
    for k in (1, 2):
        tab = brute.parity_tables(k)
        for par in (0, 1):
            want = [(drow, dcol) for kk, p, t, dcol, drow in rows
                    if kk == k and p == par]
            assert tab[par] == want


def test_golden_stride_centres():
    """Hand-worked stride examples (tests/golden/stride_centres.txt)."""
    rows = _read_rows("stride_centres.txt")
    p = 0
    while p < len(rows):
        H, W, s, Ho, Wo = rows[p]
        p += 1
        assert oracle.out_shape(H, W, s) == (Ho, Wo)
        cen = brute.lattice_centres(H, W, s)
        assert cen.shape[:2] == (Ho, Wo)
        for _ in range(Ho * Wo):
            i, j, r, c = rows[p]
            p += 1
            assert oracle.centre(i, j, s) == (r, c)
            assert tuple(cen[i, j]) == (r, c)


@pytest.mark.parametrize("s", [1, 2, 3, 4])
def test_stride_lattice_is_scaled_hex_grid(s):
    """Sec. 2.3: strides are equal steps along the three lattice axes, and
    the output keeps the hexagonal addressing -- output neighbours (as the
    addressing defines them on the output grid) sit exactly s pitches apart."""
    H, W = 30, 31
    Ho, Wo = oracle.out_shape(H, W, s)
    for i in range(1, Ho - 1):
        for j in range(1, Wo - 1):
            r0, c0 = oracle.centre(i, j, s)
            x0, y0 = _pos(r0, c0)
            for (di, dj) in _output_neighbours(j):
                r, c = oracle.centre(i + di, j + dj, s)
                x, y = _pos(r, c)
                assert abs(math.hypot(x - x0, y - y0) - s) < 1e-9


def _output_neighbours(j):
    # the six neighbours of output element (i, j), from the Sec. 2.1 layout
    # (odd columns lower): same column +-1 row, side columns rows per parity
    side = [(-1, 0), (0, 0)] if j % 2 == 0 else [(0, 0), (1, 0)]
    out = [(-1, 0), (1, 0)]
    for dj in (-1, 1):
        for di, _ in side:
            out.append((di, dj))
    return out


@pytest.mark.parametrize("H,W,s", [(40, 40, 2), (48, 48, 2), (24, 24, 2),
                                   (5, 5, 2), (7, 7, 3), (9, 10, 3),
                                   (1, 5, 2), (5, 1, 2), (2, 9, 4), (1, 1, 1),
                                   (13, 6, 5)])
def test_out_shape_matches_lattice(H, W, s):
    """Output size equals the lattice built from physical steps."""
    assert oracle.out_shape(H, W, s) == brute.lattice_centres(H, W, s).shape[:2]


# ------------------------------------------------------------ convolution

@pytest.mark.parametrize("H,W,k,s,N,Ci,Co", [
    (5, 6, 1, 1, 2, 2, 3), (7, 8, 2, 1, 1, 2, 2), (7, 7, 1, 2, 2, 1, 2),
    (9, 8, 2, 3, 1, 2, 2), (6, 9, 3, 2, 1, 1, 1), (1, 5, 1, 2, 1, 1, 1),
    (5, 1, 2, 2, 1, 1, 2), (4, 4, 0, 1, 2, 3, 2), (3, 3, 4, 1, 1, 1, 1),
    (8, 5, 1, 4, 1, 2, 1), (6, 7, 2, 2, 2, 3, 2)])
def test_conv_matches_brute_force(H, W, k, s, N, Ci, Co):
    """Whole forward definition against the physical-position brute force."""
    rng = _rng(H * 100 + W * 10 + k + s)
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, H, W))
    w = rng.normal(size=(Co, Ci, T))
    b = rng.normal(size=Co)
    y = oracle.conv_fwd(x, w, b, k, s)
    yb = brute.conv_fwd(x, w, b, k, s)
    assert y.shape == yb.shape
    np.testing.assert_allclose(y, yb, rtol=0, atol=1e-12)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_torch_conv2d_special_case(k):
    """At stride 1 the hex convolution is two dense (2k+1)^2 conv2d calls with
    parity-masked kernels (even / odd output columns)."""
    torch = pytest.importorskip("torch")
    rng = _rng(k)
    N, Ci, Co, H, W = 2, 2, 3, 9, 10
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, H, W))
    w = rng.normal(size=(Co, Ci, T))
    tab = brute.parity_tables(k)
    dense = np.zeros((2, Co, Ci, 2 * k + 1, 2 * k + 1))
    for par in (0, 1):
        for t, (drow, dcol) in enumerate(tab[par]):
            dense[par, :, :, drow + k, dcol + k] = w[:, :, t]
    xt = torch.from_numpy(x)
    out = np.zeros((N, Co, H, W))
    for par in (0, 1):
        yt = torch.nn.functional.conv2d(xt, torch.from_numpy(dense[par]),
                                        padding=k).numpy()
        out[..., par::2] = yt[..., par::2]
    np.testing.assert_allclose(oracle.conv_fwd(x, w, None, k, 1), out,
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k", [0, 1, 2, 3])
@pytest.mark.parametrize("par", [0, 1])
def test_delta_input_reproduces_kernel(k, par):
    """A single lit pixel p: the output is non-zero at exactly T pixels, and
    the output at the pixel reached from p by the reversed displacement of
    tap t equals w[t] (the hexagonal tap pattern)."""
    rng = _rng(7 + k)
    H = W = 15
    T = oracle.num_taps(k)
    w = rng.uniform(0.5, 1.5, size=(1, 1, T))
    x = np.zeros((1, 1, H, W))
    r0, c0 = 7, 6 + par
    x[0, 0, r0, c0] = 1.0
    y = oracle.conv_fwd(x, w, None, k, 1)[0, 0]
    assert np.count_nonzero(y) == T
    g = brute.Grid(H, W)
    x0, y0 = _pos(r0, c0)
    for t, (dx, dy) in enumerate(brute.kernel_offsets(k)):
        r, c = g.at(x0 - dx, y0 - dy)
        assert y[r, c] == w[0, 0, t]


@pytest.mark.parametrize("k", [1, 2, 3])
def test_constant_input(k):
    """Constant input v: interior outputs are v * sum(w) + b; every output is
    v * (sum of the weights of its in-tensor taps) + b."""
    rng = _rng(k)
    T = oracle.num_taps(k)
    w = rng.normal(size=(2, 1, T))
    b = rng.normal(size=2)
    v = 1.75
    x = np.full((1, 1, 12, 13), v)
    y = oracle.conv_fwd(x, w, b, k, 1)
    inner = y[0, :, k:-k, k:-k]
    want = v * w.sum(axis=(1, 2)) + b
    np.testing.assert_allclose(inner, want[:, None, None]
                               * np.ones_like(inner), rtol=1e-13)


def test_golden_debug_mode_all_ones():
    """Sec. 3 / Fig. 5: all kernel elements 1 -> neighbourhood counts."""
    rows = _read_rows("debug_ones_3x4_k1.txt")
    H, W, k = rows[0]
    want = np.array(rows[1:1 + H], np.float64)
    y = oracle.conv_fwd(np.ones((1, 1, H, W)), np.ones((1, 1, 7)), None, k, 1)
    np.testing.assert_array_equal(y[0, 0], want)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_all_ones_interior_count(k):
    """Debug-mode kernel on ones: interior outputs count exactly T pixels,
    border outputs fewer (padding adds nothing)."""
    T = oracle.num_taps(k)
    y = oracle.conv_fwd(np.ones((1, 1, 14, 15)), np.ones((1, 1, T)), None, k, 1)
    assert np.all(y[0, 0, k:-k, k:-k] == T)
    assert np.all(y <= T) and y.min() < T


def _rotate60(x, y):
    return (0.5 * x - SQ * y, SQ * x + 0.5 * y)


@pytest.mark.parametrize("k,s", [(1, 1), (2, 1), (1, 2), (2, 2), (1, 3)])
def test_rotation_equivariance(k, s):
    """Sec. 3: hexagonal kernels conserve 6-fold symmetry.  Rotating a
    zero-padded input by 60 degrees about a kernel centre, with the kernel
    rotated the same way, rotates the output."""
    H = W = 31
    g = brute.Grid(H, W)
    rng = _rng(k * 10 + s)
    # rotate about the centre of an output element near the middle
    Ho, Wo = oracle.out_shape(H, W, s)
    rc, cc = oracle.centre(Ho // 2, (Wo // 2) & ~1, s)
    xc, yc = _pos(rc, cc)
    R = 6.3
    x = np.zeros((1, 1, H, W))
    rot_of = {}
    for r in range(H):
        for c in range(W):
            px, py = _pos(r, c)
            if math.hypot(px - xc, py - yc) <= R:
                x[0, 0, r, c] = rng.normal()
            qx, qy = _rotate60(px - xc, py - yc)
            rot_of[(r, c)] = g.at(xc + qx, yc + qy)
    xr = np.zeros_like(x)
    for (r, c), dst in rot_of.items():
        if x[0, 0, r, c] != 0.0:
            xr[0, 0, dst[0], dst[1]] = x[0, 0, r, c]
    offs = brute.kernel_offsets(k)
    okey = {(round(a, 6), round(b, 6)): t for t, (a, b) in enumerate(offs)}
    T = len(offs)
    w = rng.normal(size=(1, 1, T))
    wr = np.zeros_like(w)
    for t, (a, b) in enumerate(offs):
        qa, qb = _rotate60(a, b)
        wr[0, 0, okey[(round(qa, 6), round(qb, 6))]] = w[0, 0, t]
    y = oracle.conv_fwd(x, w, None, k, s)[0, 0]
    yr = oracle.conv_fwd(xr, wr, None, k, s)[0, 0]
    out_at = {oracle.centre(i, j, s): (i, j)
              for i in range(Ho) for j in range(Wo)}
    checked = 0
    for (i, j) in [(i, j) for i in range(Ho) for j in range(Wo)]:
        r, c = oracle.centre(i, j, s)
        px, py = _pos(r, c)
        if math.hypot(px - xc, py - yc) > R + k + 0.5:
            continue
        dst = rot_of[(r, c)]
        assert dst is not None and dst in out_at
        i2, j2 = out_at[dst]
        assert abs(yr[i2, j2] - y[i, j]) < 1e-12
        checked += 1
    assert checked > 10
    assert np.abs(y).max() > 0


# ----------------------------------------------------------- backward pass

@pytest.mark.parametrize("k,s", [(0, 1), (1, 1), (2, 1), (1, 2), (2, 2),
                                 (3, 2), (1, 3), (2, 3), (2, 4)])
def test_bwd_data_is_adjoint(k, s):
    """dx is the adjoint of the forward map: <fwd(x), dy> = <x, bwd(dy)>."""
    rng = _rng(k + 10 * s)
    N, Ci, Co, H, W = 2, 2, 3, 11, 12
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, H, W))
    w = rng.normal(size=(Co, Ci, T))
    y = oracle.conv_fwd(x, w, None, k, s)
    dy = rng.normal(size=y.shape)
    dx = oracle.conv_bwd_data(dy, w, k, s, H, W)
    lhs = float(np.sum(y * dy))
    rhs = float(np.sum(x * dx))
    assert abs(lhs - rhs) <= 1e-11 * max(1.0, abs(lhs))


@pytest.mark.parametrize("k,s", [(1, 1), (2, 1), (1, 2), (2, 3)])
def test_bwd_weight_is_adjoint(k, s):
    """<dw, V> = <fwd_V(x), dy> for any weights V; db = sum of dy."""
    rng = _rng(3 * k + s)
    N, Ci, Co, H, W = 2, 2, 3, 10, 9
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, H, W))
    Ho, Wo = oracle.out_shape(H, W, s)
    dy = rng.normal(size=(N, Co, Ho, Wo))
    dw, db = oracle.conv_bwd_weight(x, dy, k, s)
    for _ in range(3):
        V = rng.normal(size=(Co, Ci, T))
        lhs = float(np.sum(dw * V))
        rhs = float(np.sum(oracle.conv_fwd(x, V, None, k, s) * dy))
        assert abs(lhs - rhs) <= 1e-11 * max(1.0, abs(lhs))
    np.testing.assert_allclose(db, dy.sum(axis=(0, 2, 3)), rtol=1e-13)


def test_gradients_by_finite_difference():
    """The forward map is linear in x and in w, so a finite difference of
    L = <y, dy> recovers single gradient entries up to rounding."""
    rng = _rng(99)
    N, Ci, Co, H, W, k, s = 1, 2, 2, 8, 9, 2, 2
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, H, W))
    w = rng.normal(size=(Co, Ci, T))
    b = rng.normal(size=Co)
    Ho, Wo = oracle.out_shape(H, W, s)
    dy = rng.normal(size=(N, Co, Ho, Wo))
    L = lambda xx, ww, bb: float(np.sum(oracle.conv_fwd(xx, ww, bb, k, s) * dy))
    dx = oracle.conv_bwd_data(dy, w, k, s, H, W)
    dw, db = oracle.conv_bwd_weight(x, dy, k, s)
    h = 1e-3
    for (n, ci, r, c) in [(0, 0, 4, 4), (0, 1, 0, 0), (0, 1, 7, 8), (0, 0, 3, 5)]:
        xp = x.copy()
        xp[n, ci, r, c] += h
        assert abs((L(xp, w, b) - L(x, w, b)) / h - dx[n, ci, r, c]) < 1e-8
    for (co, ci, t) in [(0, 0, 0), (1, 1, 9), (1, 0, 18)]:
        wp = w.copy()
        wp[co, ci, t] += h
        assert abs((L(x, wp, b) - L(x, w, b)) / h - dw[co, ci, t]) < 1e-8
    bp = b.copy()
    bp[1] += h
    assert abs((L(x, w, bp) - L(x, w, b)) / h - db[1]) < 1e-8


@pytest.mark.parametrize("s", [1, 2, 3])
def test_strided_equals_subsampled(s):
    """Strided output = stride-1 output read at the lattice centres (built
    from physical steps), bit for bit."""
    rng = _rng(s)
    N, Ci, Co, H, W, k = 2, 2, 2, 13, 11, 2
    T = oracle.num_taps(k)
    x = rng.normal(size=(N, Ci, H, W))
    w = rng.normal(size=(Co, Ci, T))
    b = rng.normal(size=Co)
    y1 = oracle.conv_fwd(x, w, b, k, 1)
    ys = oracle.conv_fwd(x, w, b, k, s)
    cen = brute.lattice_centres(H, W, s)
    assert ys.shape[2:] == cen.shape[:2]
    for i in range(cen.shape[0]):
        for j in range(cen.shape[1]):
            r, c = cen[i, j]
            assert np.array_equal(ys[:, :, i, j], y1[:, :, r, c])


def test_sampled_entry_points_match_full():
    """The one-element-at-a-time routines used at full size agree with the
    whole-tensor routines."""
    rng = _rng(5)
    for (N, Ci, Co, H, W, k, s) in [(2, 3, 2, 9, 10, 1, 1),
                                    (1, 2, 3, 11, 8, 2, 2),
                                    (2, 1, 2, 7, 9, 2, 3)]:
        T = oracle.num_taps(k)
        x = rng.normal(size=(N, Ci, H, W))
        w = rng.normal(size=(Co, Ci, T))
        b = rng.normal(size=Co)
        y = oracle.conv_fwd(x, w, b, k, s)
        dy = rng.normal(size=y.shape)
        idx = rng.choice(y.size, size=min(40, y.size), replace=False)
        np.testing.assert_array_equal(
            oracle.conv_fwd_at(x, w, b, k, s, idx), y.reshape(-1)[idx])
        dx = oracle.conv_bwd_data(dy, w, k, s, H, W)
        idx = rng.choice(dx.size, size=60, replace=False)
        np.testing.assert_allclose(
            oracle.conv_bwd_data_at(dy, w, k, s, H, W, idx),
            dx.reshape(-1)[idx], rtol=1e-12, atol=1e-12)
        dw, _ = oracle.conv_bwd_weight(x, dy, k, s)
        idx = rng.choice(dw.size, size=min(20, dw.size), replace=False)
        np.testing.assert_array_equal(
            oracle.conv_bwd_weight_at(x, dy, k, s, idx), dw.reshape(-1)[idx])


# ----------------------------------------------------------------- pooling

@pytest.mark.parametrize("mode", [oracle.POOL_MAX, oracle.POOL_AVG])
def test_pool_size0_is_identity(mode):
    """Sec. 2.4: pooling over a size-0 window with stride 1 returns x."""
    x = _rng(1).normal(size=(2, 3, 6, 7))
    y, am = oracle.pool_fwd(x, 0, 1, mode)
    np.testing.assert_array_equal(y, x)
    assert np.all(am == 0)


@pytest.mark.parametrize("H,W,k,s,mode", [
    (5, 6, 1, 1, 0), (7, 8, 2, 2, 0), (9, 8, 1, 2, 1), (6, 9, 2, 3, 1),
    (8, 8, 1, 2, 0), (4, 7, 3, 1, 1)])
def test_pool_matches_brute_force(H, W, k, s, mode):
    rng = _rng(H + W + k + s)
    x = rng.normal(size=(2, 2, H, W))
    x[0, 0, 1:3, 1:3] = 0.25                 # ties
    y, am = oracle.pool_fwd(x, k, s, mode)
    yb, amb = brute.pool_fwd(x, k, s, mode)
    np.testing.assert_allclose(y, yb, rtol=0, atol=1e-15)
    if mode == 0:
        np.testing.assert_array_equal(am, amb)


def test_pool_avg_constant():
    """Average of a constant v: v at interior outputs, v * (in-tensor
    taps) / T at the border (padding counts as zero, divisor T)."""
    k, s, v = 1, 2, 3.0
    H, W = 10, 10
    x = np.full((1, 1, H, W), v)
    y, _ = oracle.pool_fwd(x, k, s, oracle.POOL_AVG)
    ones = oracle.conv_fwd(np.ones((1, 1, H, W)), np.ones((1, 1, 7)), None, k, s)
    np.testing.assert_allclose(y, v * ones / 7.0, rtol=1e-15)
    assert np.any(y == v) and np.any(y < v)


def test_pool_max_ties_and_padding():
    """Max: equal values -> the first tap in canonical order wins; negative
    data at the border loses to the zero padding; non-negative data never
    reports a value below its in-tensor maximum."""
    x = np.full((1, 1, 6, 6), 2.0)
    y, am = oracle.pool_fwd(x, 1, 1, oracle.POOL_MAX)
    assert np.all(y == 2.0)
    interior = am[0, 0, 1:-1, 1:-1]
    assert np.all(interior == 0)
    xn = -np.ones((1, 1, 6, 6))
    y, _ = oracle.pool_fwd(xn, 1, 1, oracle.POOL_MAX)
    assert np.all(y[0, 0, 1:-1, 1:-1] == -1.0)
    assert y[0, 0, 0, 0] == 0.0
    xp = np.abs(_rng(2).normal(size=(1, 1, 7, 7)))
    y, _ = oracle.pool_fwd(xp, 1, 2, oracle.POOL_MAX)
    yb, _ = brute.pool_fwd(xp, 1, 2, 0)
    np.testing.assert_array_equal(y, yb)


@pytest.mark.parametrize("mode", [oracle.POOL_MAX, oracle.POOL_AVG])
@pytest.mark.parametrize("k,s", [(1, 1), (1, 2), (2, 2), (1, 3)])
def test_pool_bwd_is_adjoint(mode, k, s):
    """With the argmax fixed, both pools are linear maps y = P x; the
    gradient is P^T dy, so <P x, dy> = <x, bwd(dy)>.  With relu_y given, the
    gradient is masked to relu_y > 0."""
    rng = _rng(k * 7 + s + mode)
    N, C, H, W = 2, 2, 11, 10
    x = rng.normal(size=(N, C, H, W))
    y, am = oracle.pool_fwd(x, k, s, mode)
    dy = rng.normal(size=y.shape)
    dx = oracle.pool_bwd(dy, am if mode == 0 else None, None, k, s, mode, H, W)
    lhs, rhs = float(np.sum(y * dy)), float(np.sum(x * dx))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))
    relu_y = np.maximum(x, 0.0)
    dxm = oracle.pool_bwd(dy, am if mode == 0 else None, relu_y, k, s, mode,
                          H, W)
    np.testing.assert_array_equal(dxm, np.where(relu_y > 0, dx, 0.0))
