"""CPU oracle for the constrained parameterization and its initialization
(ResonatorLM, arXiv 2607.05583, Sec. 3.1 last paragraph).

TEST INFRASTRUCTURE ONLY.  The slow, obviously correct reference for the HIP
parameter-map kernels.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py``'s ``cpu_baseline`` leg may import it; it imports nothing from the
product path.  All arithmetic is float64.

The paper maps unconstrained parameters to the valid ranges with softplus and
sigmoid transforms, with a floor alpha_min = 1e-4 on the damping, and starts
from log-spaced half-lives and frequencies.  Readings (each also in the design
notes):
  damping     gamma = alpha_min + softplus(theta_gamma)       (gamma > alpha_min)
  frequency   omega = pi * sigmoid(theta_omega)               (0 < omega < pi)
  amplitude and phase are used as they are (no transform).
  initialization: half-lives ln 2 / gamma log-spaced from hl_min to hl_max and
  periods 2 pi / omega log-spaced from per_max down to per_min, over the M modes
  of every channel (over the D channels when M = 1, the paper's one mode per
  head).

Parity status: every function here is pinned in ``tests/test_params_oracle.py``
by closed forms (softplus(0) = ln 2, sigmoid(0) = 1/2), limits, round trips
through independently written inverses, central finite differences for the
chain rule, and the half-life / period spacing of the initialization.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = ["ALPHA_MIN", "params_map", "params_map_bwd", "params_init", "half_lives",
           "energy_decay"]

ALPHA_MIN = 1e-4


def _softplus(u):
    u = np.asarray(u, dtype=np.float64)
    return np.logaddexp(0.0, u)


def _sigmoid(u):
    """1 / (1 + e^-u), written as e^u / (1 + e^u) for u < 0 so that no exponential overflows."""
    u = np.asarray(u, dtype=np.float64)
    e = np.exp(-np.abs(u))
    return np.where(u >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def params_map(theta_gamma, theta_omega, alpha_min: float = ALPHA_MIN):
    """(gamma, omega) from unconstrained (theta_gamma, theta_omega), Sec. 3.1."""
    gamma = float(alpha_min) + _softplus(theta_gamma)
    omega = math.pi * _sigmoid(theta_omega)
    return gamma, omega


def params_map_bwd(theta_gamma, theta_omega, dgamma, domega):
    """Chain rule of ``params_map``: d/dtheta softplus = sigmoid, d/dtheta pi sigmoid
    = pi sigmoid (1 - sigmoid), written as pi sigmoid(u) sigmoid(-u) (the same value,
    without the cancellation of 1 - sigmoid for large u)."""
    sg = _sigmoid(theta_gamma)
    tw = np.asarray(theta_omega, dtype=np.float64)
    return (np.asarray(dgamma, dtype=np.float64) * sg,
            np.asarray(domega, dtype=np.float64) * math.pi * _sigmoid(tw) * _sigmoid(-tw))


def _log_spaced(lo: float, hi: float, n: int):
    if n == 1:
        return np.array([math.sqrt(lo * hi)])
    return lo * (hi / lo) ** (np.arange(n) / (n - 1))


def params_init(D: int, M: int, hl_min: float = 2.0, hl_max: float = 2048.0, per_min: float = 4.0,
                per_max: float = 2048.0, alpha_min: float = ALPHA_MIN):
    """Unconstrained (theta_gamma, theta_omega) [D, M] whose mapped values have
    log-spaced half-lives hl_min..hl_max and periods per_max..per_min over the
    modes of each channel (over the channels when M = 1)."""
    n = M if M > 1 else D
    hl = _log_spaced(hl_min, hl_max, n)                 # half-life ln2 / gamma
    per = _log_spaced(per_min, per_max, n)[::-1]        # period 2 pi / omega, long first
    gamma = math.log(2.0) / hl
    omega = np.minimum(2.0 * math.pi / per, math.pi * (1.0 - 1e-6))
    # inverses of the maps: softplus^-1(v) = log(e^v - 1), logit(p) = log(p / (1 - p))
    tg = np.log(np.expm1(gamma - alpha_min))
    p = omega / math.pi
    tw = np.log(p / (1.0 - p))
    if M > 1:
        return np.tile(tg, (D, 1)), np.tile(tw, (D, 1))
    return tg.reshape(D, 1), tw.reshape(D, 1)


def half_lives(gamma):
    """ln 2 / gamma (Sec. 3.5 diagnostics)."""
    return math.log(2.0) / np.asarray(gamma, dtype=np.float64)


def energy_decay(gamma, t):
    """State-energy decay exp(-2 gamma t) (Sec. 3.5 diagnostics): [..., len(t)]."""
    g = np.asarray(gamma, dtype=np.float64)[..., None]
    return np.exp(-2.0 * g * np.asarray(t, dtype=np.float64))


def spectrum(gamma, omega, amp, phase, T: int):
    """Magnitude of the real DFT of the length-T impulse response (Sec. 3.5
    diagnostics): |rfft(K_d[0..T-1])|, [T//2 + 1, D], with K from the direct
    kernel taps (Sec. 3.1)."""
    from .resonator_oracle import kernel_taps
    return np.abs(np.fft.rfft(kernel_taps(gamma, omega, amp, phase, T), axis=1)).T
