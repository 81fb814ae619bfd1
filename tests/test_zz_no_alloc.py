"""hexconv_bwd_noalloc (the workspace in the library's static scratch
array) against hexconv_bwd (a caller-allocated workspace) through the C
ABI: bit-identical dx, dw and db, on calls in a row whose inputs shrink, so
that later calls find the earlier calls' contents in the scratch array.
The shapes cover the three workspace users: the bf16 matrix-core weight
gradient (27.5 MiB of slot partials at the full wide layer), the fused
small-channel backward, and the generic kernels at stride 2."""
import numpy as np
import pytest

import oracle
from paper_1903_01814_amd import hexconv as hx
from paper_1903_01814_amd import inputs as gen

from gpu_helpers import check, empty, from_dev, to_dev, torch_mod

pytestmark = pytest.mark.gpu

CASES = [
    # N, Ci, Co, H, W, k, s, dtype -- in call order, each smaller than the last
    (64, 64, 64, 128, 128, 1, 1, "bf16"),
    (8, 64, 64, 64, 64, 1, 1, "bf16"),
    (16, 1, 16, 40, 40, 2, 1, "f32"),
    (2, 8, 12, 30, 31, 2, 2, "f32"),
]


def _inputs(case, seed):
    N, Ci, Co, H, W, k, s, dt = case
    rng = np.random.default_rng(seed)
    T = oracle.num_taps(k)
    Ho, Wo = oracle.out_shape(H, W, s)
    x = gen.round_to(rng.normal(size=(N, Ci, H, W)), dt)
    w = gen.round_to(rng.normal(size=(Co, Ci, T)) / np.sqrt(Ci * T), dt)
    dy = gen.round_to(rng.normal(size=(N, Co, Ho, Wo)), dt)
    return x, w, dy


def _outputs(case):
    torch = torch_mod()
    N, Ci, Co, H, W, k, s, dt = case
    T = oracle.num_taps(k)
    dx = empty((N, Ci, H, W), dt)
    dw = torch.full((Co, Ci, T), float("nan"), dtype=torch.float32, device="cuda:0")
    db = torch.full((Co,), float("nan"), dtype=torch.float32, device="cuda:0")
    return dx, dw, db


def test_noalloc_matches_bwd_on_shrinking_calls():
    torch = torch_mod()
    for i, case in enumerate(CASES):
        N, Ci, Co, H, W, k, s, dt = case
        print("noalloc case", case, flush=True)
        x, w, dy = _inputs(case, 100 + i)
        xd, wd, dyd = to_dev(x, dt), to_dev(w, dt), to_dev(dy, dt)
        dtc = hx.HEX_F32 if dt == "f32" else hx.HEX_BF16
        nws = hx.hexconv_bwd_workspace(N, Ci, Co, H, W, k, s, dtc)
        assert 0 < nws <= hx.HEX_NOALLOC_SCRATCH_BYTES
        ws = torch.empty(nws, dtype=torch.uint8, device="cuda:0")
        ref = _outputs(case)
        hx.hexconv_bwd(xd, dyd, wd, *ref, ws, k, s)
        got = _outputs(case)
        hx.hexconv_bwd_noalloc(xd, dyd, wd, *got, k, s)
        torch.cuda.synchronize()
        for name, a, b in zip(("dx", "dw", "db"), got, ref):
            assert torch.equal(a, b), "%s differs for %s" % (name, case)
        # and both meet the parity bar against the oracle (dw, db)
        if N * Ci * Co * H * W <= 4_000_000:
            rw, rb = oracle.conv_bwd_weight(x, dy, k, s)
            mw, mb = oracle.conv_bwd_weight(np.abs(x), np.abs(dy), k, s)
            check(dt, from_dev(got[1]), rw, mw, "noalloc dw")
            check(dt, from_dev(got[2]), rb, mb, "noalloc db")


def test_noalloc_without_dx():
    """dx = NULL (a first layer): weight and bias gradients only."""
    torch = torch_mod()
    case = (24, 1, 16, 40, 40, 2, 1, "bf16")
    N, Ci, Co, H, W, k, s, dt = case
    x, w, dy = _inputs(case, 7)
    xd, wd, dyd = to_dev(x, dt), to_dev(w, dt), to_dev(dy, dt)
    nws = hx.hexconv_bwd_workspace(N, Ci, Co, H, W, k, s, hx.HEX_BF16)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda:0")
    _, dw0, db0 = _outputs(case)
    hx.hexconv_bwd(xd, dyd, wd, None, dw0, db0, ws, k, s)
    _, dw1, db1 = _outputs(case)
    hx.hexconv_bwd_noalloc(xd, dyd, wd, None, dw1, db1, k, s)
    torch.cuda.synchronize()
    assert torch.equal(dw0, dw1) and torch.equal(db0, db1)
