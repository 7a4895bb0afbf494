"""Pins of the parameter-map oracle (constrained parameterization, initialization,
half-lives and energy decay; Sec. 3.1 last paragraph and Sec. 3.5).

No GPU.  Each pin is independent of the oracle's formulas: closed forms
(softplus(0) = ln 2, sigmoid(0) = 1/2), library routines (scipy's expit and
log1p / exp), inverses written here, central finite differences, and the mode
recurrence of the mixing oracle for the half-life and the energy decay.  The
last test plants plausible mistakes and checks that a pin fails.
"""
import math

import numpy as np
import pytest
from scipy.special import expit

import oracle as O
import oracle.params_oracle as P


def test_closed_forms_at_zero():
    g, w = P.params_map(np.zeros(3), np.zeros(3))
    np.testing.assert_allclose(g, P.ALPHA_MIN + math.log(2.0), rtol=0, atol=1e-15)
    np.testing.assert_allclose(w, math.pi / 2, rtol=0, atol=1e-15)


def test_against_library_routines():
    u = np.linspace(-30.0, 30.0, 241)
    g, w = P.params_map(u, u, alpha_min=0.25)
    np.testing.assert_allclose(g, 0.25 + np.log1p(np.exp(u)), rtol=1e-13, atol=1e-300)
    np.testing.assert_allclose(w, math.pi * expit(u), rtol=1e-13, atol=1e-300)


def test_ranges_and_monotonicity():
    u = np.linspace(-60.0, 60.0, 1001)
    g, w = P.params_map(u, u)
    assert np.all(g >= P.ALPHA_MIN) and np.all(g[:10] < P.ALPHA_MIN * 1.0001)
    assert np.all(w > 0.0) and np.all(w <= math.pi) and w[500] == math.pi / 2
    # non-decreasing everywhere; strictly increasing where the increments are representable
    assert np.all(np.diff(g) >= 0) and np.all(np.diff(w) >= 0)
    assert np.all(np.diff(g[u > -20]) > 0) and np.all(np.diff(w[np.abs(u) < 20]) > 0)


def test_chain_rule_by_finite_differences():
    r = np.random.default_rng(3)
    tg, tw = r.normal(scale=3.0, size=7), r.normal(scale=3.0, size=7)
    dg, dw = r.normal(size=7), r.normal(size=7)
    gg, gw = P.params_map_bwd(tg, tw, dg, dw)
    h = 1e-6
    for i in range(7):
        e = np.zeros(7)
        e[i] = h
        fd_g = (np.dot(dg, P.params_map(tg + e, tw)[0]) - np.dot(dg, P.params_map(tg - e, tw)[0])) / (2 * h)
        fd_w = (np.dot(dw, P.params_map(tg, tw + e)[1]) - np.dot(dw, P.params_map(tg, tw - e)[1])) / (2 * h)
        assert abs(gg[i] - fd_g) <= 1e-7 * max(1.0, abs(fd_g))
        assert abs(gw[i] - fd_w) <= 1e-7 * max(1.0, abs(fd_w))


@pytest.mark.parametrize("D,M", [(4, 8), (16, 1), (3, 2)])
def test_init_is_log_spaced(D, M):
    tg, tw = P.params_init(D, M)
    assert tg.shape == (D, M) and tw.shape == (D, M)
    g, w = P.params_map(tg, tw)
    n = M if M > 1 else D
    hl = (math.log(2.0) / g).reshape(-1)[:n] if M > 1 else (math.log(2.0) / g)[:, 0]
    per = (2 * math.pi / w).reshape(-1)[:n] if M > 1 else (2 * math.pi / w)[:, 0]
    # half-lives 2 .. 2048 with a constant ratio; periods 2048 .. 4 with a constant ratio
    np.testing.assert_allclose(hl[0], 2.0, rtol=1e-9)
    np.testing.assert_allclose(hl[-1], 2048.0, rtol=1e-9)
    np.testing.assert_allclose(np.diff(np.log(hl)), math.log(1024.0) / (n - 1), rtol=1e-9)
    np.testing.assert_allclose(per[0], 2048.0, rtol=1e-9)
    np.testing.assert_allclose(per[-1], 4.0, rtol=1e-9)
    if M > 1:  # every channel gets the same spread of timescales
        assert np.all(tg == tg[:1]) and np.all(tw == tw[:1])


def test_half_life_and_energy_decay_against_the_recurrence():
    """The mixing oracle's recurrence driven by a unit impulse: |h_t| = exp(-gamma t),
    so |h| halves at the half-life and |h_t|^2 is the energy decay."""
    gamma = np.array([[0.01, 0.2, 1.3]])
    omega = np.array([[0.5, 2.0, 0.1]])
    amp, phase = np.ones((1, 3)), np.zeros((1, 3))
    T = 400
    x = np.zeros((1, T, 1))
    x[0, 0, 0] = 1.0
    lam, _ = O.modes(gamma, omega, amp, phase)
    h = np.zeros(3, dtype=complex)
    mags = []
    for t in range(T):
        h = lam[0] * h + x[0, t, 0]
        mags.append(np.abs(h))
    mags = np.array(mags)  # [T, 3]
    t = np.arange(T)
    np.testing.assert_allclose(mags.T ** 2, P.energy_decay(gamma[0], t), rtol=1e-10, atol=1e-300)
    hl = P.half_lives(gamma[0])
    np.testing.assert_allclose(np.exp(-gamma[0] * hl), 0.5, rtol=1e-14)


def test_planted_mistakes_are_caught():
    """A missing floor, a missing pi and a softplus in place of the sigmoid in the
    chain rule each fail a pin above."""
    keep_map, keep_bwd = P.params_map, P.params_map_bwd

    def fails(*tests):
        for t in tests:
            try:
                t()
            except AssertionError:
                return True
        return False

    try:
        P.params_map = lambda tg, tw, alpha_min=P.ALPHA_MIN: (np.logaddexp(0, tg), math.pi * expit(tw))
        assert fails(test_closed_forms_at_zero)
        P.params_map = lambda tg, tw, alpha_min=P.ALPHA_MIN: (alpha_min + np.logaddexp(0, tg), expit(tw))
        assert fails(test_closed_forms_at_zero)
        P.params_map = keep_map
        P.params_map_bwd = lambda tg, tw, dg, dw: (dg * np.logaddexp(0, tg), dw * math.pi * expit(tw) * (1 - expit(tw)))
        assert fails(test_chain_rule_by_finite_differences)
    finally:
        P.params_map, P.params_map_bwd = keep_map, keep_bwd


def test_spectrum_against_brute_force_dft_and_the_dc_closed_form():
    """The spectrum pinned two ways: a brute-force DFT sum over the taps, written
    as a Python loop over (tau, k) for a tiny T, and the k = 0 bin in closed form
    for a single mode with a = 1, phi = 0 (the geometric sum Re (1 - lambda^T) /
    (1 - lambda))."""
    rng = np.random.default_rng(3)
    D, M, T = 3, 2, 12
    gamma = rng.uniform(0.05, 0.8, (D, M))
    omega = rng.uniform(0.1, 3.0, (D, M))
    amp = rng.uniform(-1.0, 1.0, (D, M))
    phase = rng.uniform(-3.0, 3.0, (D, M))
    S = P.spectrum(gamma, omega, amp, phase, T)
    assert S.shape == (T // 2 + 1, D)
    for d in range(D):
        K = [sum(amp[d, m] * math.exp(-gamma[d, m] * tau) * math.cos(omega[d, m] * tau + phase[d, m])
                 for m in range(M)) for tau in range(T)]
        for k in range(T // 2 + 1):
            re = sum(K[tau] * math.cos(2 * math.pi * k * tau / T) for tau in range(T))
            im = -sum(K[tau] * math.sin(2 * math.pi * k * tau / T) for tau in range(T))
            assert abs(S[k, d] - math.hypot(re, im)) <= 1e-12 * (1 + abs(S[k, d]))
    g, w = 0.3, 1.1
    lam = complex(math.exp(-g) * math.cos(w), math.exp(-g) * math.sin(w))
    dc = ((1 - lam ** T) / (1 - lam)).real
    S1 = P.spectrum(np.array([[g]]), np.array([[w]]), np.array([[1.0]]), np.array([[0.0]]), T)
    assert abs(S1[0, 0] - abs(dc)) <= 1e-12
