"""Brute-force hexagonal convolution / pooling from physical pixel positions.

TEST INFRASTRUCTURE ONLY (tiny grids).  This re-derives the whole geometry a
third way, without axial coordinates: every tensor element gets its position
in the plane, neighbours are the elements at distance one pitch, kernel taps
are found by breadth-first search over neighbour layers, and the stride
lattice is built by stepping along the lattice axes.  It checks the C oracle
(hexoracle.c), which uses axial algebra instead.

Definitions followed (HexagDLy, arXiv:1903.01814):
  * Sec. 2.1, Fig. 1: columns of vertically adjacent pixels; every second
    column shifted by half a pitch so rows line up; rows top to bottom,
    columns left to right.  Reading: odd columns lie half a pitch lower.
  * Sec. 2.2: a size-k kernel is the centre plus k layers of neighbours.
  * Sec. 2.3, Fig. 4: kernels centred on real elements only, zero padding,
    strides of equal steps along the three lattice axes from the top-left
    element, columns cut to equal length.
  * Sec. 2.4: pooling uses the same windows; max / average aggregation.
"""
from __future__ import annotations

import math
from collections import deque

import numpy as np

SQRT3_2 = math.sqrt(3.0) / 2.0
_EPS = 1e-9


def position(r: int, c: int):
    """Physical (x, y) of tensor element (r, c); y grows downwards."""
    return (c * SQRT3_2, r + 0.5 * (c & 1))


def _key(x: float, y: float):
    return (round(x / _EPS), round(y / _EPS))


def _lattice_patch(radius: int):
    """Positions of a patch of the infinite pixel lattice around (0, 0).

    Built from the addressing rule itself (a large tensor whose element
    (radius, 2*radius') is even-column), then shifted so the centre element
    sits at the origin.
    """
    n = 4 * radius + 5
    r0, c0 = n // 2, 2 * (n // 4)          # an even column
    x0, y0 = position(r0, c0)
    pts = []
    for r in range(n):
        for c in range(n):
            x, y = position(r, c)
            pts.append((x - x0, y - y0))
    return pts


def kernel_offsets(k: int):
    """Physical displacement vectors of the taps of a size-k kernel.

    Layers of neighbours found by breadth-first search over elements at
    distance one pitch; returned in canonical order (x ascending, then y
    ascending, i.e. column by column, each top to bottom).
    """
    pts = _lattice_patch(k + 2)
    index = {_key(x, y): p for p, (x, y) in enumerate(pts)}
    origin = index[_key(0.0, 0.0)]
    # neighbours: the six elements at unit distance (found by search)
    unit = []
    for (x, y) in pts:
        d = math.hypot(x, y)
        if abs(d - 1.0) < 1e-9:
            unit.append((x, y))
    assert len(unit) == 6, unit
    layer = {origin: 0}
    q = deque([origin])
    while q:
        p = q.popleft()
        if layer[p] == k:
            continue
        x, y = pts[p]
        for (ux, uy) in unit:
            nb = index.get(_key(x + ux, y + uy))
            if nb is not None and nb not in layer:
                layer[nb] = layer[p] + 1
                q.append(nb)
    offs = [pts[p] for p in layer]
    offs.sort(key=lambda v: (round(v[0] / _EPS), round(v[1] / _EPS)))
    return offs


def unit_steps():
    """The six unit neighbour vectors."""
    return [v for v in kernel_offsets(1) if math.hypot(*v) > 0.5]


class Grid:
    """Position lookup for an H x W tensor."""

    def __init__(self, H: int, W: int):
        self.H, self.W = H, W
        self.where = {}
        for r in range(H):
            for c in range(W):
                self.where[_key(*position(r, c))] = (r, c)

    def at(self, x: float, y: float):
        return self.where.get(_key(x, y))


def lattice_centres(H: int, W: int, stride: int):
    """Kernel centres under the hex-preserving stride, as an (Ho, Wo) array
    of (r, c) tensor elements.

    Centres are reached from the top-left element by steps of `stride`
    pitches along the lattice axes; those that land on tensor elements are
    grouped into columns (same x), each sorted top to bottom, and every
    column is cut to the length of the shortest one.
    """
    g = Grid(H, W)
    ux, uy = 0.0, 1.0                       # straight down a column
    vx, vy = SQRT3_2, 0.5                   # down-right diagonal
    span = H + W + 2
    # lattice columns: every multiple of `stride` columns to the right of the
    # top-left element that still lies inside the tensor (possibly holding
    # no centre at all when H is small)
    col_x = []
    b = 0
    while stride * b * vx < (W - 0.5) * SQRT3_2:
        col_x.append(stride * b * vx)
        b += 1
    cols = {bx: [] for bx in range(len(col_x))}
    for a in range(-span, span + 1):
        for bx in range(len(col_x)):
            x = stride * (a * ux + bx * vx)
            y = stride * (a * uy + bx * vy)
            rc = g.at(x, y)
            if rc is not None:
                cols[bx].append(rc)
    keys = sorted(cols)
    if not keys:
        return np.zeros((0, 0, 2), np.int64)
    ho = min(len(cols[c]) for c in keys)
    out = np.zeros((ho, len(keys), 2), np.int64)
    for j, c in enumerate(keys):
        col = sorted(cols[c])
        for i in range(ho):
            out[i, j] = col[i]
    return out


def _windows(H, W, k, stride):
    """For every output (i, j): list of input elements (or None) per tap."""
    g = Grid(H, W)
    offs = kernel_offsets(k)
    cen = lattice_centres(H, W, stride)
    Ho, Wo = cen.shape[:2]
    win = []
    for i in range(Ho):
        row = []
        for j in range(Wo):
            r, c = cen[i, j]
            x, y = position(int(r), int(c))
            row.append([g.at(x + dx, y + dy) for (dx, dy) in offs])
        win.append(row)
    return win, Ho, Wo, len(offs)


def conv_fwd(x, w, b, k, stride=1):
    x = np.asarray(x, np.float64)
    N, Ci, H, W = x.shape
    Co = w.shape[0]
    win, Ho, Wo, T = _windows(H, W, k, stride)
    assert w.shape == (Co, Ci, T)
    y = np.zeros((N, Co, Ho, Wo))
    for n in range(N):
        for co in range(Co):
            for i in range(Ho):
                for j in range(Wo):
                    acc = 0.0 if b is None else float(b[co])
                    for ci in range(Ci):
                        for t, e in enumerate(win[i][j]):
                            if e is not None:
                                acc += w[co, ci, t] * x[n, ci, e[0], e[1]]
                    y[n, co, i, j] = acc
    return y


def pool_fwd(x, k, stride, mode):
    """mode 0 = max (first maximal tap, padding counts as 0), 1 = average."""
    x = np.asarray(x, np.float64)
    N, C, H, W = x.shape
    win, Ho, Wo, T = _windows(H, W, k, stride)
    y = np.zeros((N, C, Ho, Wo))
    am = np.zeros((N, C, Ho, Wo), np.int32)
    for n in range(N):
        for ch in range(C):
            for i in range(Ho):
                for j in range(Wo):
                    vals = [0.0 if e is None else x[n, ch, e[0], e[1]]
                            for e in win[i][j]]
                    if mode == 0:
                        best = max(vals)
                        am[n, ch, i, j] = vals.index(best)
                        y[n, ch, i, j] = best
                    else:
                        y[n, ch, i, j] = sum(vals) / T
    return y, am


def parity_tables(k):
    """(drow, dcol) of every tap for an even and an odd centre column,
    found by locating the physical displacement from a centre element."""
    offs = kernel_offsets(k)
    H = W = 4 * k + 6
    g = Grid(H, W)
    out = {}
    for par in (0, 1):
        r0, c0 = 2 * k + 2, 2 * k + 2 + par
        x0, y0 = position(r0, c0)
        tab = []
        for (dx, dy) in offs:
            r, c = g.at(x0 + dx, y0 + dy)
            tab.append((r - r0, c - c0))
        out[par] = tab
    return out


# ------------------------------------------------------------ three dimensions
# Sec. 2.4: hexagonal x-y planes, equidistant samples along z.  Here the z
# axis is modelled as its own equidistant lattice: plane d sits at height d;
# the window of a centre plane z0 holds the planes at heights z0 - kz ..
# z0 + kz that exist (others read zero), and the centres are reached by
# steps of stride_z from the first plane.

def z_centres(D: int, stride_z: int):
    out, z = [], 0
    while z < D:
        out.append(z)
        z += stride_z
    return out


def conv3d_fwd(x, w, b, k, kz, stride=1, stride_z=1):
    x = np.asarray(x, np.float64)
    N, Ci, D, H, W = x.shape
    Co = w.shape[0]
    win, Ho, Wo, T = _windows(H, W, k, stride)
    zc = z_centres(D, stride_z)
    assert w.shape == (Co, Ci, 2 * kz + 1, T)
    y = np.zeros((N, Co, len(zc), Ho, Wo))
    for n in range(N):
        for co in range(Co):
            for l, z0 in enumerate(zc):
                for i in range(Ho):
                    for j in range(Wo):
                        acc = 0.0 if b is None else float(b[co])
                        for ci in range(Ci):
                            for h in range(-kz, kz + 1):
                                if not 0 <= z0 + h < D:
                                    continue
                                for t, e in enumerate(win[i][j]):
                                    if e is not None:
                                        acc += w[co, ci, h + kz, t] * x[n, ci, z0 + h, e[0], e[1]]
                        y[n, co, l, i, j] = acc
    return y


def pool3d_fwd(x, k, kz, stride, stride_z, mode):
    """mode 0 = max (value of the first maximal tap, planes in ascending
    height, padding counts as 0), 1 = average over all (2kz+1) T taps."""
    x = np.asarray(x, np.float64)
    N, C, D, H, W = x.shape
    win, Ho, Wo, T = _windows(H, W, k, stride)
    zc = z_centres(D, stride_z)
    y = np.zeros((N, C, len(zc), Ho, Wo))
    am = np.zeros(y.shape, np.int32)
    for n in range(N):
        for ch in range(C):
            for l, z0 in enumerate(zc):
                for i in range(Ho):
                    for j in range(Wo):
                        vals = []
                        for h in range(-kz, kz + 1):
                            for e in win[i][j]:
                                inside = e is not None and 0 <= z0 + h < D
                                vals.append(x[n, ch, z0 + h, e[0], e[1]] if inside else 0.0)
                        if mode == 0:
                            best = max(vals)
                            am[n, ch, l, i, j] = vals.index(best)
                            y[n, ch, l, i, j] = best
                        else:
                            y[n, ch, l, i, j] = sum(vals) / len(vals)
    return y, am
