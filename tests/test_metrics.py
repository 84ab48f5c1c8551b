"""CPU pins of the image-quality measurements (PSNR, SSIM) reported beside
the frame rate: closed forms, identities and a window-by-window brute force
on tiny images."""
import math

import numpy as np
import torch

from paper_2607_03390_amd import metrics as M


def test_psnr_closed_form():
    x = torch.full((3, 8, 9), 0.3, dtype=torch.float32)
    assert abs(M.psnr(x + 0.1, x) - 20.0) < 1e-5    # MSE 0.01
    assert M.psnr(x, x) == math.inf
    # clamping to [0, 1]: values above 1 count as 1
    assert abs(M.psnr(torch.full_like(x, 2.0), torch.full_like(x, 0.9)) - 20.0) < 1e-5


def test_ssim_identity_and_symmetry():
    g = torch.Generator().manual_seed(0)
    x = torch.rand((3, 32, 40), generator=g)
    y = (x + 0.1 * torch.randn((3, 32, 40), generator=g)).clamp(0, 1)
    assert abs(M.ssim(x, x) - 1.0) < 1e-12
    assert abs(M.ssim(x, y) - M.ssim(y, x)) < 1e-12
    assert M.ssim(x, y) < 0.99


def test_ssim_constant_images_closed_form():
    # zero variance and covariance: SSIM = (2ab + C1) / (a^2 + b^2 + C1)
    for a, b in ((0.2, 0.7), (0.5, 0.5), (0.0, 1.0)):
        x = torch.full((3, 16, 16), a, dtype=torch.float64)
        y = torch.full((3, 16, 16), b, dtype=torch.float64)
        want = (2 * a * b + M.C1) / (a * a + b * b + M.C1)
        assert abs(M.ssim(x, y) - want) < 1e-12


def test_ssim_bruteforce_windows():
    # every window position of a tiny image, weighted sums written out
    rng = np.random.default_rng(1)
    x = rng.random((2, 13, 12))
    y = np.clip(x + 0.2 * rng.standard_normal(x.shape), 0, 1)
    t = np.arange(M.WINDOW) - (M.WINDOW - 1) / 2
    g1 = np.exp(-t * t / (2 * M.SIGMA ** 2))
    w = np.outer(g1, g1)
    w /= w.sum()
    vals = []
    for c in range(2):
        for i in range(13 - M.WINDOW + 1):
            for j in range(12 - M.WINDOW + 1):
                px = x[c, i:i + M.WINDOW, j:j + M.WINDOW]
                py = y[c, i:i + M.WINDOW, j:j + M.WINDOW]
                mx, my = (w * px).sum(), (w * py).sum()
                vx = (w * (px - mx) ** 2).sum()
                vy = (w * (py - my) ** 2).sum()
                cxy = (w * (px - mx) * (py - my)).sum()
                vals.append((2 * mx * my + M.C1) * (2 * cxy + M.C2) /
                            ((mx * mx + my * my + M.C1) * (vx + vy + M.C2)))
    assert abs(M.ssim(torch.from_numpy(x), torch.from_numpy(y)) - float(np.mean(vals))) < 1e-12
