"""Physics diagnostics of a resonant mode bank (Sec. 3.5), as a library utility.

They read the parameters, not attention maps:

- ``half_lives``: ln 2 / gamma per mode, and ``energy_decay``: exp(-2 gamma t)
  per mode (library kernel, float64 inside);
- ``spectrum``: the magnitude of the real DFT of the length-T impulse response,
  evaluated in closed form per mode by the library (a geometric sum per bin in
  float64, no impulse response or FFT needed);
- ``impulse_response``: the kernel K_d[tau] for tau < T, produced by the mixing
  kernels themselves on a unit impulse;
- ``causality_check``: perturbs the suffix of an input and reports the largest
  change of the output prefix (the paper reports below 1e-6; the chunked scan
  here gives exactly 0, as no prefix output reads a later input).
"""
from __future__ import annotations

import torch

from . import _lib, ops


def _params(*ts):
    for t in ts:
        if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or not t.is_cuda or t.shape != ts[0].shape:
            raise ValueError("parameters must be float32 device tensors of one shape [D, M]")
        if not t.is_contiguous():
            raise ValueError("parameters must be contiguous")


def _diag(gamma, omega, amp, phase, T, hl=False, en=False, sp=False):
    D, M = gamma.shape
    h = torch.empty((D, M), dtype=torch.float32, device=gamma.device) if hl else None
    e = torch.empty((D, M, T), dtype=torch.float32, device=gamma.device) if en else None
    s = torch.empty((T // 2 + 1, D), dtype=torch.float32, device=gamma.device) if sp else None
    p = lambda t: ops._ptr(t) if t is not None else None
    ops.check(_lib.lib().resonator_diagnostics(p(gamma), p(omega), p(amp), p(phase), D, M, T, p(h), p(e), p(s),
                                               ops._stream(gamma.device)))
    return h, e, s


def half_lives(gamma: torch.Tensor) -> torch.Tensor:
    """ln 2 / gamma, [D, M]."""
    _params(gamma)
    return _diag(gamma, None, None, None, 1, hl=True)[0]


def energy_decay(gamma: torch.Tensor, T: int) -> torch.Tensor:
    """exp(-2 gamma t) for t = 0 .. T-1: [D, M, T]."""
    _params(gamma)
    return _diag(gamma, None, None, None, T, en=True)[1]


def spectrum(gamma, omega, amp, phase, T: int) -> torch.Tensor:
    """|real DFT| of the length-T impulse response: [T // 2 + 1, D]."""
    _params(gamma, omega, amp, phase)
    return _diag(gamma, omega, amp, phase, T, sp=True)[2]


def impulse_response(gamma, omega, amp, phase, T: int) -> torch.Tensor:
    """K_d[tau], tau < T, [T, D] float32: the mixing of a unit impulse at t = 0."""
    D = gamma.shape[0]
    x = torch.zeros((1, T, D), dtype=torch.float32, device=gamma.device)
    x[:, 0, :] = 1.0
    return ops.resonator_mix_fwd(x, gamma, omega, amp, phase)[0]


def causality_check(x: torch.Tensor, gamma, omega, amp, phase, split: int, scale: float = 1.0) -> float:
    """Largest |y'[:, :split] - y[:, :split]| when x[:, split:] is replaced by noise."""
    y = ops.resonator_mix_fwd(x, gamma, omega, amp, phase)
    xp = x.clone()
    g = torch.Generator(device=x.device).manual_seed(0)
    noise = torch.randn(xp[:, split:].shape, generator=g, device=x.device, dtype=torch.float32) * scale
    xp[:, split:] = noise.to(x.dtype)
    yp = ops.resonator_mix_fwd(xp, gamma, omega, amp, phase)
    return float((yp[:, :split].float() - y[:, :split].float()).abs().max()) if split > 0 else 0.0
