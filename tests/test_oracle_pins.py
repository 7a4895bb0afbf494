"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests needs a GPU.  Each pin is independent of the oracle's own
formulas: exact hand-derived fixtures (tests/golden/), closed forms, a library
routine (scipy.signal.lfilter, numpy.cumsum, numpy.convolve), brute force and
finite differences.  ``test_planted_mistakes_are_caught`` plants plausible
mistakes on the oracle side and checks that some pin fails for each.
"""
import math

import numpy as np
import pytest

import oracle as O
from golden_util import load, value
from workloads import random_problem

P4 = ("gamma", "omega", "amp", "phase")


def params_of(prob):
    return tuple(prob[k] for k in P4)


def single_mode(alpha, omega, phi, a=1.0, D=1):
    f = lambda v: np.full((D, 1), v, dtype=np.float64)
    return f(alpha), f(omega), f(a), f(phi)


# --------------------------------------------------------------------------
# exact fixtures
# --------------------------------------------------------------------------
def _impulse(n):
    x = np.zeros((1, n, 1))
    x[0, 0, 0] = 1.0
    return x


@pytest.mark.parametrize("case", range(4))
def test_golden_kernel_all_forms(case):
    c = load("kernel_exact.json")["cases"][case]
    exp = np.array([value(s) for s in c["k"]])
    prm = single_mode(value(c["alpha"]), value(c["omega"]), value(c["phi"]))
    n = len(exp)
    np.testing.assert_allclose(O.kernel_taps(*prm, n)[0], exp, atol=1e-15)
    x = _impulse(n)
    for form in (O.mix_direct, O.mix_fft, O.mix_lfilter):
        np.testing.assert_allclose(form(x, *prm)[0, :, 0], exp, atol=1e-14)
    np.testing.assert_allclose(O.mix_recurrence(x, *prm)[0][0, :, 0], exp, atol=1e-15)


def test_golden_decode_states_and_outputs():
    g = load("decode_exact.json")
    u = np.array([value(s) for s in g["u"]])
    sre = np.array([value(s) for s in g["state_re"]])
    sim = np.array([value(s) for s in g["state_im"]])
    for c in g["cases"]:
        prm = single_mode(value(g["alpha"]), value(g["omega"]), value(c["phi"]), a=value(c["a"]))
        exp = np.array([value(s) for s in c["y"]])
        # decode, one drive per call
        state = np.zeros((1, 1, 1, 2))
        for t in range(len(u)):
            y, state = O.decode_step(state, np.array([[u[t]]]), *prm)
            assert abs(y[0, 0] - exp[t]) < 1e-14
            assert abs(state[0, 0, 0, 0] - sre[t]) < 1e-14
            assert abs(state[0, 0, 0, 1] - sim[t]) < 1e-14
        x = u.reshape(1, -1, 1)
        np.testing.assert_allclose(O.mix_direct(x, *prm)[0, :, 0], exp, atol=1e-14)
        yr, hl = O.mix_recurrence(x, *prm)
        np.testing.assert_allclose(yr[0, :, 0], exp, atol=1e-14)
        np.testing.assert_allclose(hl[0, 0, 0], [sre[-1], sim[-1]], atol=1e-14)
        np.testing.assert_allclose(O.state_init(x, *prm)[0, 0, 0], [sre[-1], sim[-1]], atol=1e-14)


def test_golden_half_life():
    g = load("half_life.json")
    for hl in g["half_lives"]:
        n = int(2 * hl) + 1
        prm = single_mode(math.log(2.0) / hl, 0.0, 0.0)
        k = O.kernel_taps(*prm, n)[0]
        assert abs(k[int(hl)] - value(g["expected_at_half_life"])) < 1e-12
        assert abs(k[int(2 * hl)] - value(g["expected_at_twice"])) < 1e-12


# --------------------------------------------------------------------------
# closed forms and library routines
# --------------------------------------------------------------------------
def test_impulse_response_random_params():
    prob = random_problem(11, 1, 40, 5, 3)
    prm = params_of(prob)
    K = O.kernel_taps(*prm, 40)
    x = np.zeros((1, 40, 5))
    x[0, 0, :] = 1.0
    for y in (O.mix_direct(x, *prm), O.mix_recurrence(x, *prm)[0], O.mix_fft(x, *prm),
              O.mix_lfilter(x, *prm)):
        np.testing.assert_allclose(y[0].T, K, atol=1e-13)


def test_constant_input_geometric_closed_form():
    prob = random_problem(12, 2, 64, 4, 3)
    prm = params_of(prob)
    lam = np.exp(-np.asarray(prm[0], np.float64)) * np.exp(1j * np.asarray(prm[1], np.float64))
    c = np.asarray(prm[2], np.float64) * np.exp(1j * np.asarray(prm[3], np.float64))
    t = np.arange(64)[:, None, None]
    # sum_{k=0..t} lambda^k = (1 - lambda^(t+1)) / (1 - lambda), written with numpy's power
    exp = (c[None] * (1 - np.power(lam[None], t + 1)) / (1 - lam[None])).real.sum(-1)  # [L, D]
    x = np.ones((2, 64, 4))
    for y in (O.mix_direct(x, *prm), O.mix_recurrence(x, *prm)[0], O.mix_fft(x, *prm),
              O.mix_lfilter(x, *prm)):
        np.testing.assert_allclose(y[0], exp, rtol=1e-11, atol=1e-12)
        np.testing.assert_allclose(y[1], exp, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("seed,B,L,D,M", [(1, 2, 33, 3, 2), (2, 1, 70, 4, 5), (3, 3, 17, 2, 8)])
def test_four_forms_agree_bruteforce(seed, B, L, D, M):
    prob = random_problem(seed, B, L, D, M, gamma_range=(1e-4, 1.0), gamma_log=True)
    prm = params_of(prob)
    x = prob["x"]
    yd = O.mix_direct(x, *prm)
    scale = np.abs(yd).max()
    for y in (O.mix_recurrence(x, *prm)[0], O.mix_fft(x, *prm), O.mix_lfilter(x, *prm)):
        assert np.abs(y - yd).max() <= 1e-12 * scale
    pos = np.array([[b, t, d] for b in range(B) for t in (0, L // 2, L - 1) for d in range(D)])
    np.testing.assert_allclose(O.mix_direct_at(x, *prm, pos), yd[pos[:, 0], pos[:, 1], pos[:, 2]],
                               rtol=1e-12, atol=1e-12 * scale)


def test_undamped_dc_mode_is_cumsum():
    D, M = 3, 4
    rng = np.random.default_rng(5)
    a = rng.normal(size=(D, M))
    ph = rng.uniform(0, 2 * np.pi, size=(D, M))
    z = np.zeros((D, M))
    x = rng.normal(size=(2, 50, D))
    exp = np.cumsum(x, axis=1) * (a * np.cos(ph)).sum(1)[None, None, :]
    for y in (O.mix_direct(x, z, z, a, ph), O.mix_recurrence(x, z, z, a, ph)[0], O.mix_fft(x, z, z, a, ph)):
        np.testing.assert_allclose(y, exp, rtol=1e-12, atol=1e-12)


def test_heavy_damping_is_memoryless():
    D, M = 3, 4
    rng = np.random.default_rng(6)
    a, ph, w = rng.normal(size=(D, M)), rng.uniform(0, 6, size=(D, M)), rng.uniform(0, 3, size=(D, M))
    g = np.full((D, M), 60.0)
    x = rng.normal(size=(1, 30, D))
    exp = x * (a * np.cos(ph)).sum(1)[None, None, :]
    for y in (O.mix_direct(x, g, w, a, ph), O.mix_recurrence(x, g, w, a, ph)[0]):
        np.testing.assert_allclose(y, exp, rtol=1e-12, atol=1e-14)


def test_paper_head_case_matches_numpy_convolve():
    """Sec. 3.1/3.2: one mode per head, amplitude 1, shared by the head's d_h channels.

    H = 2 heads of d_h = 32 channels (D = 64); y_h = k_h * u_h per channel via
    numpy.convolve truncated to the causal part.
    """
    H, dh, L = 2, 32, 48
    rng = np.random.default_rng(7)
    alpha = rng.uniform(1e-3, 0.5, size=H)
    om = rng.uniform(0, np.pi, size=H)
    ph = rng.uniform(0, 2 * np.pi, size=H)
    g = np.repeat(alpha, dh)[:, None]
    w = np.repeat(om, dh)[:, None]
    p = np.repeat(ph, dh)[:, None]
    a = np.ones((H * dh, 1))
    u = rng.normal(size=(1, L, H * dh))
    y = O.mix_recurrence(u, g, w, a, p)[0]
    tt = np.arange(L)
    for h in range(H):
        k = np.exp(-alpha[h] * tt) * np.cos(om[h] * tt + ph[h])
        for j in range(dh):
            d = h * dh + j
            np.testing.assert_allclose(y[0, :, d], np.convolve(k, u[0, :, d])[:L], atol=1e-12)


def test_linearity_shift_invariance_causality():
    prob = random_problem(8, 2, 64, 3, 4, gamma_range=(1e-4, 1.0), gamma_log=True)
    prm = params_of(prob)
    rng = np.random.default_rng(9)
    x1, x2 = rng.normal(size=(2, 64, 3)), rng.normal(size=(2, 64, 3))
    f = lambda x: O.mix_recurrence(x, *prm)[0]
    np.testing.assert_allclose(f(2.5 * x1 - 0.75 * x2), 2.5 * f(x1) - 0.75 * f(x2), rtol=1e-11, atol=1e-11)
    xs = np.zeros_like(x1)
    xs[:, 10:] = x1[:, :-10]
    np.testing.assert_allclose(f(xs)[:, 10:], f(x1)[:, :-10], rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(f(xs)[:, :10], 0.0)
    # causality (Sec. 3.5): perturbing the suffix leaves the prefix exactly unchanged
    xp = x1.copy()
    xp[:, 40:] += rng.normal(size=(2, 24, 3))
    for form in (O.mix_recurrence, O.mix_direct):
        ya = form(x1, *prm)
        yb = form(xp, *prm)
        ya = ya[0] if isinstance(ya, tuple) else ya
        yb = yb[0] if isinstance(yb, tuple) else yb
        assert np.array_equal(ya[:, :40], yb[:, :40])
        assert np.abs(ya[:, 40:] - yb[:, 40:]).max() > 1e-3


# --------------------------------------------------------------------------
# state, decode, split prefill
# --------------------------------------------------------------------------
def test_state_energy_decay():
    """Sec. 3.5: under zero drive the state energy decays as exp(-2 alpha t)."""
    prob = random_problem(10, 2, 1, 3, 4, with_h0=True)
    prm = params_of(prob)
    s = prob["h0"].astype(np.float64)
    e0 = (s ** 2).sum(-1)
    for t in range(1, 30):
        _, s = O.decode_step(s, np.zeros((2, 3)), *prm)
        np.testing.assert_allclose((s ** 2).sum(-1), e0 * np.exp(-2 * prm[0].astype(np.float64) * t)[None],
                                   rtol=1e-12)


def test_prefill_then_decode_equals_full_sequence():
    prob = random_problem(13, 2, 60, 4, 3, gamma_range=(1e-4, 1.0), gamma_log=True)
    prm = params_of(prob)
    x = prob["x"].astype(np.float64)
    L0 = 37
    full = O.mix_direct(x, *prm)
    st = O.state_init(x[:, :L0], *prm)
    np.testing.assert_allclose(st, O.mix_recurrence(x[:, :L0], *prm)[1], rtol=1e-12, atol=1e-12)
    ys, st2 = O.decode_run(st, np.transpose(x[:, L0:], (1, 0, 2)), *prm)
    np.testing.assert_allclose(np.transpose(ys, (1, 0, 2)), full[:, L0:], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(st2, O.state_init(x, *prm), rtol=1e-11, atol=1e-11)
    assert np.array_equal(O.state_init(x[:, :0], *prm), np.zeros((2, 4, 3, 2)))


def test_split_prefill_with_initial_state():
    prob = random_problem(14, 2, 50, 3, 5, with_h0=True, gamma_range=(1e-4, 1.0), gamma_log=True)
    prm = params_of(prob)
    x, h0 = prob["x"].astype(np.float64), prob["h0"].astype(np.float64)
    y_full, h_full = O.mix_recurrence(x, *prm, h0=h0)
    y1, h1 = O.mix_recurrence(x[:, :21], *prm, h0=h0)
    y2, h2 = O.mix_recurrence(x[:, 21:], *prm, h0=h1)
    np.testing.assert_allclose(np.concatenate([y1, y2], 1), y_full, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(h2, h_full, rtol=1e-12, atol=1e-12)
    # the direct form writes the h0 term with exact arguments, independently of the recurrence
    np.testing.assert_allclose(O.mix_direct(x, *prm, h0=h0), y_full, rtol=1e-11, atol=1e-11)
    pos = np.array([[1, 0, 2], [0, 49, 1], [1, 33, 0]])
    np.testing.assert_allclose(O.mix_direct_at(x, *prm, pos, h0=h0), y_full[pos[:, 0], pos[:, 1], pos[:, 2]],
                               rtol=1e-11, atol=1e-11)


# --------------------------------------------------------------------------
# backward
# --------------------------------------------------------------------------
def _loss(x, dy, g, w, a, p, h0):
    return float((O.mix_direct(x, g, w, a, p, h0=h0) * dy).sum())


def test_bwd_matches_central_differences():
    prob = random_problem(15, 2, 14, 3, 2, with_h0=True, with_dy=True, gamma_range=(1e-2, 0.8))
    x, dy, h0 = (prob[k].astype(np.float64) for k in ("x", "dy", "h0"))
    prm = [prob[k].astype(np.float64) for k in P4]
    gr = O.mix_bwd(x, dy, *prm, h0=h0)
    eps = 1e-6
    names = {"gamma": "dgamma", "omega": "domega", "amp": "damp", "phase": "dphase"}
    for i, k in enumerate(P4):
        num = np.zeros_like(prm[i])
        for idx in np.ndindex(*prm[i].shape):
            pp = [q.copy() for q in prm]
            pm = [q.copy() for q in prm]
            pp[i][idx] += eps
            pm[i][idx] -= eps
            num[idx] = (_loss(x, dy, *pp, h0) - _loss(x, dy, *pm, h0)) / (2 * eps)
        np.testing.assert_allclose(gr[names[k]], num, rtol=1e-7, atol=1e-7)
    for name, arr in (("dx", x), ("dh0", h0)):
        num = np.zeros_like(arr)
        for idx in list(np.ndindex(*arr.shape))[::5]:
            ap, am = arr.copy(), arr.copy()
            ap[idx] += eps
            am[idx] -= eps
            if name == "dx":
                num[idx] = (_loss(ap, dy, *prm, h0) - _loss(am, dy, *prm, h0)) / (2 * eps)
            else:
                num[idx] = (_loss(x, dy, *prm, ap) - _loss(x, dy, *prm, am)) / (2 * eps)
            assert abs(gr[name][idx] - num[idx]) < 1e-7 * max(1.0, abs(num[idx]))


def test_bwd_matches_direct_kernel_derivative():
    prob = random_problem(16, 2, 40, 3, 4, with_dy=True, gamma_range=(1e-4, 1.0), gamma_log=True)
    prm = params_of(prob)
    gr = O.mix_bwd(prob["x"], prob["dy"], *prm)
    gd = O.mix_bwd_direct(prob["x"], prob["dy"], *prm)
    for k in ("damp", "dphase", "dgamma", "domega"):
        np.testing.assert_allclose(gr[k], gd[k], rtol=1e-10, atol=1e-10 * np.abs(gd[k]).max())


def test_bwd_dx_is_time_reversed_forward():
    """The transpose of a causal Toeplitz operator is the time-reversed operator."""
    prob = random_problem(17, 2, 45, 3, 4, with_dy=True, gamma_range=(1e-4, 1.0), gamma_log=True)
    prm = params_of(prob)
    dx = O.mix_bwd(prob["x"], prob["dy"], *prm)["dx"]
    rev = O.mix_direct(prob["dy"][:, ::-1], *prm)[:, ::-1]
    np.testing.assert_allclose(dx, rev, rtol=1e-11, atol=1e-11)


def test_bwd_amplitude_and_phase_identities():
    """y is linear in c = a e^{i phi}: da_m = <dy, y(a := e_m)>, dphi_m = <dy, y(a := a_m e_m, phi_m + pi/2)>."""
    prob = random_problem(18, 2, 30, 2, 3, with_dy=True)
    g, w, a, p = (prob[k].astype(np.float64) for k in P4)
    x, dy = prob["x"], prob["dy"]
    gr = O.mix_bwd(x, dy, g, w, a, p)
    for d in range(2):
        for m in range(3):
            e = np.zeros_like(a)
            e[d, m] = 1.0
            da = (O.mix_direct(x, g, w, e, p) * dy).sum()
            assert abs(gr["damp"][d, m] - da) < 1e-10 * max(1, abs(da))
            e2 = e * a[d, m]
            p2 = p.copy()
            p2[d, m] += np.pi / 2
            dp = (O.mix_direct(x, g, w, e2, p2) * dy).sum()
            assert abs(gr["dphase"][d, m] - dp) < 1e-10 * max(1, abs(dp))


# --------------------------------------------------------------------------
# planted mistakes (on the oracle side, CPU only) must be caught by the pins
# --------------------------------------------------------------------------
def _golden_decode_ok(step_fn):
    g = load("decode_exact.json")
    u = [value(s) for s in g["u"]]
    for c in g["cases"]:
        prm = single_mode(value(g["alpha"]), value(g["omega"]), value(c["phi"]), a=value(c["a"]))
        state = np.zeros((1, 1, 1, 2))
        for t in range(len(u)):
            y, state = step_fn(state, np.array([[u[t]]]), *prm)
            if abs(y[0, 0] - value(c["y"][t])) > 1e-12:
                return False
    return True


def test_planted_mistakes_are_caught():
    assert _golden_decode_ok(O.decode_step)
    # readout with c = a e^{-i phi} (the decode equation's printed sign)
    wrong_sign = lambda s, x, g, w, a, p: O.decode_step(s, x, g, w, a, -p)
    assert not _golden_decode_ok(wrong_sign)
    # conjugated pole (omega sign)
    conj_pole = lambda s, x, g, w, a, p: O.decode_step(s, x, g, -w, a, p)
    assert not _golden_decode_ok(conj_pole)

    # dropped lag 0: output read before the current drive enters
    def no_lag0(s, x, g, w, a, p):
        y, s2 = O.decode_step(s, np.zeros_like(x), g, w, a, p)
        _, s3 = O.decode_step(s, x, g, w, a, p)
        return y, s3
    assert not _golden_decode_ok(no_lag0)

    # a sign error in dgamma, or a transposed lag (t - s -> s - t) in dx, fails the brute-force pins
    prob = random_problem(19, 1, 20, 2, 2, with_dy=True)
    prm = params_of(prob)
    gr = O.mix_bwd(prob["x"], prob["dy"], *prm)
    gd = O.mix_bwd_direct(prob["x"], prob["dy"], *prm)
    assert not np.allclose(-gr["dgamma"], gd["dgamma"], rtol=1e-6)
    causal_dx = O.mix_direct(prob["dy"], *prm)           # forgot the time reversal
    assert not np.allclose(causal_dx, gr["dx"], rtol=1e-6)
