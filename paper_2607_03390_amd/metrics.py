"""Image-quality measurements of a rendered frame against a reference frame.

The paper reports PSNR, SSIM and LPIPS (Sec. IV-A, metrics).  Here they
compare a TemporalGS frame with the full render of the same camera (PSNR and
SSIM; LPIPS needs pretrained network weights and is not computed).  These are
measurements of the hot path's output, not part of it: plain PyTorch on
whatever device the images live on.

PSNR: 10 log10(1 / MSE) over all channels and pixels of images clamped to
[0, 1].  SSIM: the structural similarity index of Wang, Bovik, Sheikh and
Simoncelli (IEEE TIP 2004) with the usual constants: an 11 x 11 Gaussian
window of standard deviation 1.5, C1 = (0.01 L)^2, C2 = (0.03 L)^2, L = 1,
evaluated where the window fits inside the image and averaged over those
positions and the three channels.
"""
from __future__ import annotations

import math

import torch

WINDOW = 11
SIGMA = 1.5
C1 = 0.01 ** 2
C2 = 0.03 ** 2


def psnr(img: torch.Tensor, ref: torch.Tensor) -> float:
    """PSNR in dB of two [C, H, W] images clamped to [0, 1] (inf if equal)."""
    mse = torch.mean((img.clamp(0, 1).double() - ref.clamp(0, 1).double()) ** 2).item()
    return math.inf if mse == 0.0 else -10.0 * math.log10(mse)


def _window(device) -> torch.Tensor:
    x = torch.arange(WINDOW, dtype=torch.float64, device=device) - (WINDOW - 1) / 2.0
    g = torch.exp(-(x * x) / (2.0 * SIGMA * SIGMA))
    return g / g.sum()


def _blur(x: torch.Tensor, g: torch.Tensor) -> torch.Tensor:
    """Separable Gaussian filter, 'valid' positions only; x: [C, 1, H, W]."""
    x = torch.nn.functional.conv2d(x, g.view(1, 1, 1, WINDOW))
    return torch.nn.functional.conv2d(x, g.view(1, 1, WINDOW, 1))


def ssim(img: torch.Tensor, ref: torch.Tensor) -> float:
    """Mean SSIM of two [C, H, W] images clamped to [0, 1] (computed in fp64
    on the CPU, in fp32 on a GPU, where the filtering runs as convolutions)."""
    if img.shape != ref.shape or img.dim() != 3:
        raise ValueError("ssim expects two [C, H, W] images of the same shape")
    if img.shape[1] < WINDOW or img.shape[2] < WINDOW:
        raise ValueError(f"ssim needs images of at least {WINDOW} x {WINDOW} pixels")
    dt = torch.float64 if img.device.type == "cpu" else torch.float32
    x = img.clamp(0, 1).to(dt).unsqueeze(1)
    y = ref.clamp(0, 1).to(dt).unsqueeze(1)
    g = _window(x.device).to(dt)
    mx, my = _blur(x, g), _blur(y, g)
    sxx = _blur(x * x, g) - mx * mx
    syy = _blur(y * y, g) - my * my
    sxy = _blur(x * y, g) - mx * my
    num = (2.0 * mx * my + C1) * (2.0 * sxy + C2)
    den = (mx * mx + my * my + C1) * (sxx + syy + C2)
    return float((num / den).mean().item())
