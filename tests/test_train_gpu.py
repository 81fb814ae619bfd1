"""End-to-end training through the autograd layers: a synthetic analogue of
the paper's toy study (Sec. 4), hexagonal CNN side only.

Four shapes that keep the grid's 6-fold structure (a filled hexagon, a
hexagonal ring, a triangle and a straight line along an axial direction)
are drawn at random positions on a 16x16 hexagonal grid in offset-column
layout and overlaid with Gaussian noise; a small h-CNN (two hexagonal
convolutions with fused ReLU and max pooling, a global maximum over
positions, three fully connected layers, about 8k parameters) is trained on
128 images per class and must classify a fresh test set.  The shapes and
the network are this test's own choices: the paper's figures and notebook
are not available.
"""
import numpy as np
import pytest

from gpu_helpers import torch_mod

pytestmark = pytest.mark.gpu

H = W = 16
NOISE = 0.3


def _axial_cells(shape):
    """Cells (dq, ds) of a shape around its centre, in axial steps."""
    cells = []
    for dq in range(-3, 4):
        for ds in range(-3, 4):
            d = max(abs(dq), abs(ds), abs(dq + ds))
            if shape == 0 and d <= 2:                     # filled hexagon
                cells.append((dq, ds))
            elif shape == 1 and d == 2:                   # hexagonal ring
                cells.append((dq, ds))
            elif shape == 2 and dq >= -1 and ds >= -1 and dq + ds <= 1:  # triangle
                cells.append((dq, ds))
    if shape == 3:                                        # line along q
        cells = [(dq, 0) for dq in range(-2, 3)]
    return cells


def _images(n_per_class, rng):
    """Images [4 n, 1, H, W] float32 and labels; offset-column layout with
    odd columns shifted down (axial (q, s) = (c, r - floor(c / 2)))."""
    xs, ys = [], []
    for shape in range(4):
        cells = _axial_cells(shape)
        for _ in range(n_per_class):
            img = rng.normal(0.0, NOISE, size=(H, W))
            r0 = int(rng.integers(3, H - 3))
            c0 = int(rng.integers(3, W - 3))
            s0 = r0 - c0 // 2
            for dq, ds in cells:
                c = c0 + dq
                r = s0 + ds + c // 2
                img[r, c] += 1.0
            xs.append(img)
            ys.append(shape)
    x = np.stack(xs)[:, None].astype(np.float32)
    return x, np.array(ys, np.int64)


def test_hex_cnn_learns_shapes():
    torch = torch_mod()
    hn = pytest.importorskip("paper_1903_01814_amd.nn")
    torch.manual_seed(0)
    rng = np.random.default_rng(0)
    dev = "cuda:0"
    xtr, ytr = _images(128, rng)
    xte, yte = _images(64, rng)

    class GlobalMax(torch.nn.Module):
        # the shapes sit anywhere on the grid: classify from the strongest
        # response of each feature map
        def forward(self, x):
            return torch.amax(x, dim=(2, 3))

    net = torch.nn.Sequential(
        hn.HexConv2d(1, 16, 2, relu=True, device=dev),             # radius-2 hexagons
        hn.HexMaxPool2d(1, 2),                                     # 16x16 -> 8x8
        hn.HexConv2d(16, 32, 1, relu=True, device=dev),
        hn.HexMaxPool2d(1, 2),                                     # 8x8 -> 4x4
        GlobalMax(),
        torch.nn.Linear(32, 64), torch.nn.ReLU(),
        torch.nn.Linear(64, 32), torch.nn.ReLU(),
        torch.nn.Linear(32, 4)).to(dev)
    nparam = sum(p.numel() for p in net.parameters())
    assert 5_000 < nparam < 20_000
    opt = torch.optim.Adam(net.parameters(), lr=3e-3)
    xt = torch.from_numpy(xtr).to(dev)
    yt = torch.from_numpy(ytr).to(dev)
    losses = []
    for epoch in range(60):
        perm = torch.from_numpy(rng.permutation(len(ytr))).to(dev)
        tot = 0.0
        for i in range(0, len(ytr), 64):
            idx = perm[i:i + 64]
            loss = torch.nn.functional.cross_entropy(net(xt[idx]), yt[idx])
            opt.zero_grad()
            loss.backward()
            opt.step()
            tot += float(loss.detach()) * len(idx)
        losses.append(tot / len(ytr))
    with torch.no_grad():
        pred = net(torch.from_numpy(xte).to(dev)).argmax(1).cpu().numpy()
    acc = float((pred == yte).mean())
    print("h-CNN: %d parameters, loss %.3f -> %.4f, test accuracy %.3f"
          % (nparam, losses[0], losses[-1], acc))
    assert losses[-1] < 0.25 * losses[0]
    assert acc >= 0.95, "test accuracy %.3f" % acc
