"""Shared helpers for the GPU parity tests: device transfer and the
tolerance checks (relative L2 for float32, error over the magnitude sum of
the contributing terms for bfloat16)."""
import numpy as np
import pytest

import oracle

F32_REL_L2 = 1e-5     # float32 paths: ||gpu - ref||_2 / ||ref||_2
BF16_REL_MAG = 1e-2   # bf16 paths: |gpu - ref| / sum|terms| per element


def torch_mod():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch


def tdtype(dt):
    torch = torch_mod()
    return torch.float32 if dt == "f32" else torch.bfloat16


def to_dev(a, dt):
    """float64 numpy (values exact in dt) -> device tensor of dtype dt."""
    torch = torch_mod()
    t = torch.from_numpy(np.ascontiguousarray(a, np.float64))
    return t.to(tdtype(dt)).contiguous().to("cuda:0")


def from_dev(t):
    return t.detach().float().cpu().double().numpy()


def empty(shape, dt):
    torch = torch_mod()
    return torch.full(shape, float("nan"), dtype=tdtype(dt), device="cuda:0")


def rel_l2(got, ref):
    got = np.asarray(got, np.float64).ravel()
    ref = np.asarray(ref, np.float64).ravel()
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    return num / den if den > 0 else num


def check_f32(got, ref, what=""):
    assert np.all(np.isfinite(got)), what + ": non-finite values"
    e = rel_l2(got, ref)
    assert e <= F32_REL_L2, "%s: rel-L2 %.3g > %g" % (what, e, F32_REL_L2)
    return e


def check_bf16(got, ref, mag, what=""):
    """|got - ref| <= 1e-2 * mag element-wise; mag = sum of |term| of each
    element's sum (elements with mag 0 must be exactly 0)."""
    got = np.asarray(got, np.float64).ravel()
    ref = np.asarray(ref, np.float64).ravel()
    mag = np.asarray(mag, np.float64).ravel()
    assert np.all(np.isfinite(got)), what + ": non-finite values"
    err = np.abs(got - ref)
    zero = mag == 0
    assert np.all(err[zero] == 0), what + ": non-zero where all terms vanish"
    ratio = np.max(err[~zero] / mag[~zero]) if np.any(~zero) else 0.0
    assert ratio <= BF16_REL_MAG, "%s: max err/mag %.3g > %g" % (
        what, ratio, BF16_REL_MAG)
    return ratio


def check(dt, got, ref, mag, what=""):
    if dt == "f32":
        return check_f32(got, ref, what)
    return check_bf16(got, ref, mag, what)


def round_bf16_f64(a):
    from paper_1903_01814_amd.inputs import round_bf16
    return round_bf16(a)


def bf16_ulp(a):
    """Spacing of bfloat16 numbers at |a| (for |a| in the normal range)."""
    a = np.abs(np.asarray(a, np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, 2.0 ** (e - 7), 2.0 ** -133)


def sample_indices(shape, n, rng, edges=True):
    """Random flat indices into an NCHW tensor plus, if edges, every element
    of the first and last row and column of the first and last image
    (ragged tiles and borders)."""
    N, C, H, W = shape
    idx = set(rng.choice(N * C * H * W, size=min(n, N * C * H * W),
                         replace=False).tolist())
    if edges:
        for nn in {0, N - 1}:
            for c in {0, C - 1}:
                base = (nn * C + c) * H * W
                for w in range(W):
                    idx.add(base + w)
                    idx.add(base + (H - 1) * W + w)
                for h in range(H):
                    idx.add(base + h * W)
                    idx.add(base + h * W + W - 1)
    return np.array(sorted(idx), np.int64)


def oracle_fwd_at(x, w, b, k, s, idx):
    ref = oracle.conv_fwd_at(x, w, b, k, s, idx)
    mag = oracle.conv_fwd_at(np.abs(x), np.abs(w),
                             None if b is None else np.abs(b), k, s, idx)
    return ref, mag
