"""Physics diagnostics of a resonant mode bank (Sec. 3.5), as a library utility.

They read the parameters, not attention maps:

- ``impulse_response``: the kernel K_d[tau] for tau < T, produced by the mixing
  kernels themselves on a unit impulse;
- ``spectrum``: the magnitude of the FFT of that impulse response;
- ``half_lives``: ln 2 / gamma per mode;
- ``energy_decay``: exp(-2 gamma t) per mode;
- ``causality_check``: perturbs the suffix of an input and reports the largest
  change of the output prefix (the paper reports below 1e-6; the chunked scan
  here gives exactly 0, as no prefix output reads a later input).

The closed forms and the FFT are small elementwise or library operations on the
parameter bank and one impulse response; the mixing itself always runs through
the HIP kernels.
"""
from __future__ import annotations

import math

import torch

from . import ops


def half_lives(gamma: torch.Tensor) -> torch.Tensor:
    """ln 2 / gamma, [D, M]."""
    return math.log(2.0) / gamma


def energy_decay(gamma: torch.Tensor, T: int) -> torch.Tensor:
    """exp(-2 gamma t) for t = 0 .. T-1: [D, M, T]."""
    t = torch.arange(T, dtype=gamma.dtype, device=gamma.device)
    return torch.exp(-2.0 * gamma[..., None] * t)


def impulse_response(gamma, omega, amp, phase, T: int) -> torch.Tensor:
    """K_d[tau], tau < T, [T, D] float32: the mixing of a unit impulse at t = 0."""
    D = gamma.shape[0]
    x = torch.zeros((1, T, D), dtype=torch.float32, device=gamma.device)
    x[:, 0, :] = 1.0
    return ops.resonator_mix_fwd(x, gamma, omega, amp, phase)[0]


def spectrum(impulse: torch.Tensor) -> torch.Tensor:
    """|FFT| of an impulse response [T, D] along time: [T // 2 + 1, D]."""
    return torch.fft.rfft(impulse, dim=0).abs()


def causality_check(x: torch.Tensor, gamma, omega, amp, phase, split: int, scale: float = 1.0) -> float:
    """Largest |y'[:, :split] - y[:, :split]| when x[:, split:] is replaced by noise."""
    y = ops.resonator_mix_fwd(x, gamma, omega, amp, phase)
    xp = x.clone()
    g = torch.Generator(device=x.device).manual_seed(0)
    noise = torch.randn(xp[:, split:].shape, generator=g, device=x.device, dtype=torch.float32) * scale
    xp[:, split:] = noise.to(x.dtype)
    yp = ops.resonator_mix_fwd(xp, gamma, omega, amp, phase)
    return float((yp[:, :split].float() - y[:, :split].float()).abs().max()) if split > 0 else 0.0
