"""CPU oracle for causal resonant field mixing (ResonatorLM, arXiv 2607.05583).

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct reference
that the HIP path is checked against.  Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it; the product path
(``paper_2607_05583_amd``) never imports, calls or links anything here, and this
module imports nothing from the product path.

All arithmetic is float64 (complex128).  Inputs are taken as given: float32
parameters and float32 / bfloat16 activations convert exactly to float64.

Notation (per channel d, mode m, time t):
  damping gamma > 0, frequency omega, phase phi, amplitude a;
  lambda = exp(-gamma) (cos omega + i sin omega)           (Sec. 3.3, decay factor)
  c      = a (cos phi + i sin phi)                          (Sec. 3.1 phase sign)
  K_d[tau] = sum_m a exp(-gamma tau) cos(omega tau + phi)   (Sec. 3.1, kernel eq.)
  y[b,t,d] = sum_{s<=t} K_d[t-s] x[b,s,d]                   (Sec. 3.2, causal conv eq.)
           + Re sum_m c lambda^(t+1) h0[b,d,m]              (initial state, if any)
The recurrence form h_t = lambda h_{t-1} + x_t, y_t = Re sum_m c h_t with
h_{-1} = h0 is the same operator (Sec. 3.3, decode recurrence).

Readings of the paper that this oracle fixes (each also listed in the design
notes): the readout uses c = a e^{+i phi} so that decode reproduces the kernel
cos(omega t + phi) (the decode equation prints e^{-i phi}); lag 0 is included;
the terminal state gives the newest drive weight 1; the paper's single mode per
head with unit amplitude is the case M = 1, a = 1 of the per-channel bank.

Every function states the passage it follows.  The backward formulas are derived
here from the kernel equation (the paper trains through autograd and prints no
gradient); the derivation is in ``mix_bwd``'s docstring.

Parity status: every function below is pinned by the CPU tests in
``tests/test_oracle_pins.py`` (closed forms, exact hand-derived fixtures in
``tests/golden/``, library routines, brute force, finite differences).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "as_f64", "modes", "kernel_taps", "mix_direct", "mix_direct_at",
    "mix_recurrence", "mix_fft", "mix_lfilter", "state_init", "decode_step",
    "decode_run", "mix_bwd", "mix_bwd_direct", "bf16_bits_to_f64",
]


def as_f64(a) -> np.ndarray:
    """Exact conversion of float32/float64 input to float64."""
    return np.asarray(a, dtype=np.float64)


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact value of bfloat16 numbers given as their uint16 bit patterns."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def modes(gamma, omega, amp, phase):
    """Per-mode pole and readout coefficient, arrays [D, M] -> complex128 [D, M].

    lambda = exp(-gamma) (cos omega + i sin omega)   -- Sec. 3.3, decay-factor eq.
    c      = a (cos phi + i sin phi)                 -- readout matching the
             kernel cos(omega t + phi) of Sec. 3.1 (phase-sign reading).
    """
    g, w, a, p = (as_f64(v) for v in (gamma, omega, amp, phase))
    lam = np.exp(-g) * (np.cos(w) + 1j * np.sin(w))
    c = a * (np.cos(p) + 1j * np.sin(p))
    return lam, c


def _lam_pow(gamma, omega, k):
    """lambda^k evaluated directly as exp(k(-gamma + i omega)); k broadcastable."""
    g, w = as_f64(gamma), as_f64(omega)
    k = as_f64(k)
    return np.exp(-g * k) * (np.cos(w * k) + 1j * np.sin(w * k))


def kernel_taps(gamma, omega, amp, phase, n: int) -> np.ndarray:
    """K_d[tau] for tau = 0..n-1, shape [D, n].

    Sec. 3.1, kernel equation k[t] = exp(-alpha t) cos(omega t + phi) for lag
    t >= 0, summed over the channel's M modes with amplitude a.  Evaluated
    directly (no powers, no recurrence).
    """
    g, w, a, p = (as_f64(v)[..., None] for v in (gamma, omega, amp, phase))
    tau = np.arange(n, dtype=np.float64)
    return (a * np.exp(-g * tau) * np.cos(w * tau + p)).sum(axis=1)


def _h0_term(gamma, omega, amp, phase, h0, L):
    """Re sum_m c lambda^(t+1) h0 for t = 0..L-1, shape [B, L, D]; h0 [B, D, M, 2].

    Written out with cos/sin of the exact arguments: c lambda^(t+1) has modulus
    a e^{-gamma(t+1)} and angle omega (t+1) + phi.
    """
    h0 = as_f64(h0)
    g, w, a, p = (as_f64(v) for v in (gamma, omega, amp, phase))
    k = np.arange(1, L + 1, dtype=np.float64)[:, None, None]          # [L,1,1]
    env = a[None] * np.exp(-g[None] * k)                               # [L,D,M]
    ang = w[None] * k + p[None]
    re, im = env * np.cos(ang), env * np.sin(ang)                      # [L,D,M]
    # Re((re + i im)(h_re + i h_im)) = re h_re - im h_im
    return (np.einsum("tdm,bdm->btd", re, h0[..., 0])
            - np.einsum("tdm,bdm->btd", im, h0[..., 1]))


def mix_direct(x, gamma, omega, amp, phase, h0=None) -> np.ndarray:
    """Direct O(L^2) causal sum, y[b,t,d] = sum_{s<=t} K_d[t-s] x[b,s,d] (+ h0 term).

    Sec. 3.2, causal convolution eq. y_h = k_h * u_h with the kernel of Sec. 3.1.
    x: [B, L, D] float; params [D, M]; h0 optional [B, D, M, 2] (re, im).
    """
    x = as_f64(x)
    B, L, D = x.shape
    K = kernel_taps(gamma, omega, amp, phase, L)                       # [D, L]
    y = np.empty_like(x)
    for t in range(L):
        # sum_s K[:, t-s] x[:, s, :] for s = 0..t
        y[:, t, :] = np.einsum("bsd,ds->bd", x[:, : t + 1, :], K[:, t::-1])
    if h0 is not None:
        y += _h0_term(gamma, omega, amp, phase, h0, L)
    return y


def mix_direct_at(x, gamma, omega, amp, phase, positions, h0=None) -> np.ndarray:
    """y at selected (b, t, d) positions by the direct sum, O(t M) each.

    Same definition as ``mix_direct`` (Sec. 3.1 kernel, Sec. 3.2 causal conv);
    used to spot-check outputs at sizes where the full O(L^2) sum is too slow.
    positions: int array [P, 3] of (b, t, d).
    """
    x = as_f64(x)
    g, w, a, p = (as_f64(v) for v in (gamma, omega, amp, phase))
    pos = np.asarray(positions, dtype=np.int64)
    out = np.empty(len(pos), dtype=np.float64)
    for i, (b, t, d) in enumerate(pos):
        tau = np.arange(t + 1, dtype=np.float64)
        taps = (a[d][:, None] * np.exp(-g[d][:, None] * tau)
                * np.cos(w[d][:, None] * tau + p[d][:, None])).sum(axis=0)
        out[i] = np.dot(taps, x[b, t::-1, d])
        if h0 is not None:
            k = t + 1.0
            env = a[d] * np.exp(-g[d] * k)
            ang = w[d] * k + p[d]
            hh = as_f64(h0)[b, d]
            out[i] += np.sum(env * np.cos(ang) * hh[:, 0] - env * np.sin(ang) * hh[:, 1])
    return out


def mix_recurrence(x, gamma, omega, amp, phase, h0=None):
    """Sequential complex recurrence; returns (y [B,L,D], h_last [B,D,M,2]).

    Sec. 3.3 recurrence s_{t+1} = lambda s_t + u_t, read out with c (phase
    reading) and including the current drive (lag 0):
        h_t = lambda h_{t-1} + x_t,  h_{-1} = h0 (default 0),  y_t = Re sum_m c h_t.
    h_last = h_{L-1} is the terminal state used to continue decoding (Sec. 3.2,
    cache construction after prefill).
    """
    x = as_f64(x)
    B, L, D = x.shape
    lam, c = modes(gamma, omega, amp, phase)
    M = lam.shape[1]
    h = np.zeros((B, D, M), dtype=np.complex128)
    if h0 is not None:
        h0 = as_f64(h0)
        h = h0[..., 0] + 1j * h0[..., 1]
    y = np.empty((B, L, D), dtype=np.float64)
    for t in range(L):
        h = lam[None] * h + x[:, t, :, None]
        y[:, t, :] = (c[None] * h).real.sum(axis=-1)
    return y, np.stack([h.real, h.imag], axis=-1)


def mix_fft(x, gamma, omega, amp, phase) -> np.ndarray:
    """FFT evaluation of the causal convolution (Sec. 3.2, FFT equation).

    y = F^-1(F(u) . F(k)) with zero padding to a power of two.  The padded length
    is the next power of two >= 2L so that the circular convolution equals the
    linear (causal) one on the first L outputs (reading of "next power of two").
    """
    x = as_f64(x)
    B, L, D = x.shape
    n = 1
    while n < 2 * L:
        n *= 2
    K = kernel_taps(gamma, omega, amp, phase, L)                       # [D, L]
    X = np.fft.rfft(x, n=n, axis=1)
    Kf = np.fft.rfft(K.T, n=n, axis=0)                                 # [n/2+1, D]
    return np.fft.irfft(X * Kf[None], n=n, axis=1)[:, :L, :]


def mix_lfilter(x, gamma, omega, amp, phase) -> np.ndarray:
    """Each mode as a real second-order IIR filter run by ``scipy.signal.lfilter``.

    The mode's transfer function Re-part of c / (1 - lambda z^-1) for real input
    is (b0 + b1 z^-1) / (1 + a1 z^-1 + a2 z^-2) with
        b0 = a cos phi,  b1 = -a e^{-gamma} cos(phi - omega),
        a1 = -2 e^{-gamma} cos omega,  a2 = e^{-2 gamma}.
    A textbook-routine form of the Sec. 3.1 kernel (its impulse response is
    a e^{-gamma t} cos(omega t + phi)).  Zero initial state only.
    """
    from scipy.signal import lfilter

    x = as_f64(x)
    g, w, a, p = (as_f64(v) for v in (gamma, omega, amp, phase))
    B, L, D = x.shape
    y = np.zeros_like(x)
    for d in range(D):
        for m in range(g.shape[1]):
            num = [a[d, m] * np.cos(p[d, m]),
                   -a[d, m] * np.exp(-g[d, m]) * np.cos(p[d, m] - w[d, m])]
            den = [1.0, -2.0 * np.exp(-g[d, m]) * np.cos(w[d, m]), np.exp(-2.0 * g[d, m])]
            y[:, :, d] += lfilter(num, den, x[:, :, d], axis=1)
    return y


def state_init(x, gamma, omega, amp, phase) -> np.ndarray:
    """Terminal state after a prompt, [B, D, M, 2] (re, im).

    Sec. 3.2, cache construction: terminal state h_{L-1} = sum_s lambda^(L-1-s) x_s,
    every past drive scaled by the pole raised to its age (newest drive weight 1;
    reading of the terminal-state index).  Powers are
    evaluated directly from their exact integer lags.  L = 0 gives the zero state.
    """
    x = as_f64(x)
    B, L, D = x.shape
    M = as_f64(gamma).shape[1]
    if L == 0:
        return np.zeros((B, D, M, 2))
    lags = np.arange(L - 1, -1, -1, dtype=np.float64)[:, None, None]  # [L,1,1]
    w = _lam_pow(np.asarray(gamma)[None], np.asarray(omega)[None], lags)  # [L,D,M]
    h = np.einsum("bsd,sdm->bdm", x, w)
    return np.stack([h.real, h.imag], axis=-1)


def decode_step(state, x_t, gamma, omega, amp, phase):
    """One recurrent decode step (Sec. 3.3): h <- lambda h + x_t, y_t = Re sum_m c h.

    state [B, D, M, 2], x_t [B, D]; returns (y_t [B, D], new state [B, D, M, 2]).
    """
    lam, c = modes(gamma, omega, amp, phase)
    s = as_f64(state)
    h = s[..., 0] + 1j * s[..., 1]
    h = lam[None] * h + as_f64(x_t)[..., None]
    y = (c[None] * h).real.sum(axis=-1)
    return y, np.stack([h.real, h.imag], axis=-1)


def decode_run(state, xs, gamma, omega, amp, phase):
    """Apply ``decode_step`` to xs [T, B, D] in order; returns (ys [T, B, D], state)."""
    xs = as_f64(xs)
    ys = np.empty(xs.shape, dtype=np.float64)
    s = as_f64(state)
    for t in range(xs.shape[0]):
        ys[t], s = decode_step(s, xs[t], gamma, omega, amp, phase)
    return ys, s


def mix_bwd(x, dy, gamma, omega, amp, phase, h0=None):
    """Gradients of sum(dy * y) for y = mix(x; gamma, omega, a, phi, h0).

    Derived from the Sec. 3.1 kernel (the paper prints no backward).  With
    h_t = lambda h_{t-1} + x_t (h_{-1} = h0) and y_t = Re sum_m c h_t:
      * dx_s = sum_{t>=s} K[t-s] dy_t = Re sum_m c q_s, where the adjoint state
        q_s = lambda q_{s+1} + dy_s runs backwards from q_L = 0.
      * y is linear in c = a e^{i phi}:  W = sum_{b,t} dy_t h_t  gives
        da = Re(e^{i phi} W),  dphi = -Im(c W).
      * d lambda^k / d gamma = -k lambda^k,  d lambda^k / d omega = i k lambda^k,
        so with the lag-weighted state r_t = sum_s (t-s) lambda^(t-s) x_s
        (+ (t+1) lambda^(t+1) h0), obeying r_t = lambda r_{t-1} + lambda h_{t-1},
        and R = sum dy_t r_t:  dgamma = -Re(c R),  domega = -Im(c R).
      * y_t depends on h0 through Re(c lambda^(t+1) h0), so
        dh0 = (Re(c lambda q_0), -Im(c lambda q_0)).
    Returns a dict of float64 arrays: dx [B,L,D], dgamma/domega/damp/dphase [D,M],
    dh0 [B,D,M,2].
    """
    x, dy = as_f64(x), as_f64(dy)
    B, L, D = x.shape
    lam, c = modes(gamma, omega, amp, phase)
    M = lam.shape[1]
    h = np.zeros((B, D, M), dtype=np.complex128)
    if h0 is not None:
        h0a = as_f64(h0)
        h = h0a[..., 0] + 1j * h0a[..., 1]
    r = np.zeros_like(h)
    W = np.zeros((D, M), dtype=np.complex128)
    R = np.zeros((D, M), dtype=np.complex128)
    for t in range(L):
        r = lam[None] * r + lam[None] * h
        h = lam[None] * h + x[:, t, :, None]
        W += np.einsum("bd,bdm->dm", dy[:, t, :], h)
        R += np.einsum("bd,bdm->dm", dy[:, t, :], r)
    q = np.zeros((B, D, M), dtype=np.complex128)
    dx = np.empty_like(x)
    for s in range(L - 1, -1, -1):
        q = lam[None] * q + dy[:, s, :, None]
        dx[:, s, :] = (c[None] * q).real.sum(axis=-1)
    e_iphi = np.exp(1j * as_f64(phase))
    cq = c[None] * lam[None] * q                                   # q is q_0 here
    return {
        "dx": dx,
        "damp": (e_iphi * W).real,
        "dphase": -(c * W).imag,
        "dgamma": -(c * R).real,
        "domega": -(c * R).imag,
        "dh0": np.stack([cq.real, -cq.imag], axis=-1),
    }


def mix_bwd_direct(x, dy, gamma, omega, amp, phase):
    """Parameter gradients by differentiating the Sec. 3.1 kernel term by term.

    O(L^2) per channel, zero initial state; for tiny shapes only.  With
    e = exp(-gamma tau):  dK/da = e cos(omega tau + phi),
    dK/dphi = -a e sin(.),  dK/dgamma = -tau a e cos(.),  dK/domega = -tau a e sin(.);
    each gradient is sum_{b, s<=t} dy[b,t,d] x[b,s,d] dK/dtheta[t-s].
    """
    x, dy = as_f64(x), as_f64(dy)
    g, w, a, p = (as_f64(v) for v in (gamma, omega, amp, phase))
    B, L, D = x.shape
    tau = np.arange(L, dtype=np.float64)
    # C[d, tau] = sum_{b, s} x[b, s, d] dy[b, s + tau, d]
    C = np.zeros((D, L))
    for k in range(L):
        C[:, k] = np.einsum("bsd,bsd->d", x[:, : L - k, :], dy[:, k:, :])
    e = np.exp(-g[..., None] * tau)                                  # [D,M,L]
    ang = w[..., None] * tau + p[..., None]
    cosv, sinv = np.cos(ang), np.sin(ang)
    Cb = C[:, None, :]
    return {
        "damp": (Cb * e * cosv).sum(-1),
        "dphase": (Cb * (-a[..., None]) * e * sinv).sum(-1),
        "dgamma": (Cb * (-tau) * a[..., None] * e * cosv).sum(-1),
        "domega": (Cb * (-tau) * a[..., None] * e * sinv).sum(-1),
    }
