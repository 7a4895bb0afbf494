"""Pins of the mixer-epilogue oracle (head coupling, gate, local path; Sec. 3.4).

No GPU.  Each pin is independent of the oracle's formulas: the reductions of the
paper's equations to a library routine (lambda_c = 0 and K = 0 leave the gate
alone: scipy.special.expit), brute-force loops over the convolution and the
head sum, the impulse response of the local path, head-permutation
equivariance, and central finite differences for the backward.  The last test
plants plausible mistakes in a copy of the oracle and checks that a pin fails.
"""
import numpy as np
import pytest
from scipy.special import expit

import oracle as O


def problem(B=2, L=9, H=3, dh=2, K=3, seed=0):
    r = np.random.default_rng(seed)
    D = H * dh
    return dict(y=r.normal(size=(B, L, D)), gate=r.normal(size=(B, L, D)), v=r.normal(size=(B, L, D)),
                dz=r.normal(size=(B, L, D)), Ct=r.normal(size=(H, H)), lambda_c=0.7,
                w=r.normal(size=(D, K)) if K else np.zeros((D, 0)), s=r.normal(size=D), H=H)


def fwd(p, **over):
    q = {**p, **over}
    return O.epilogue_fwd(q["y"], q["gate"], q["v"], q["Ct"], q["lambda_c"], q["w"], q["s"], q["H"])


def test_uncoupled_gate_only_is_sigmoid_times_y():
    p = problem(K=0)
    z = fwd(p, lambda_c=0.0)
    np.testing.assert_allclose(z, expit(p["gate"]) * p["y"], rtol=1e-14, atol=1e-14)


def test_identity_coupling_when_ct_is_zero():
    p = problem(K=0)
    np.testing.assert_allclose(O.coupling_matrix(np.zeros((4, 4)), 3.0), np.eye(4), atol=0)
    z = fwd(p, Ct=np.zeros_like(p["Ct"]))
    np.testing.assert_allclose(z, expit(p["gate"]) * p["y"], rtol=1e-14, atol=1e-14)


def test_coupling_against_loops():
    p = problem(K=0, seed=3)
    B, L, D = p["y"].shape
    H, dh = p["H"], D // p["H"]
    C = np.eye(H) + p["lambda_c"] / np.sqrt(H) * np.tanh(p["Ct"])
    ref = np.zeros((B, L, D))
    for b in range(B):
        for t in range(L):
            for g in range(H):
                for j in range(dh):
                    acc = 0.0
                    for h in range(H):
                        acc += C[g, h] * p["y"][b, t, h * dh + j]
                    ref[b, t, g * dh + j] = expit(p["gate"][b, t, g * dh + j]) * acc
    np.testing.assert_allclose(fwd(p), ref, rtol=1e-12, atol=1e-12)


def test_local_path_impulse_response():
    """A unit drive at (b, t0, c) with y = 0 gives z[b, t0 + k, c] = s[c] w[c, k], else 0."""
    p = problem(K=4, seed=5)
    B, L, D = p["y"].shape
    v = np.zeros((B, L, D))
    b, t0, c = 1, 2, 4
    v[b, t0, c] = 1.0
    z = fwd(p, y=np.zeros((B, L, D)), v=v)
    ref = np.zeros((B, L, D))
    for k in range(4):
        if t0 + k < L:
            ref[b, t0 + k, c] = p["s"][c] * p["w"][c, k]
    np.testing.assert_allclose(z, ref, atol=1e-15)


def test_local_path_is_causal_and_matches_numpy_convolve():
    p = problem(K=3, seed=6)
    B, L, D = p["y"].shape
    z = fwd(p, y=np.zeros((B, L, D)))
    for b in range(B):
        for c in range(D):
            ref = p["s"][c] * np.convolve(p["v"][b, :, c], p["w"][c])[:L]
            np.testing.assert_allclose(z[b, :, c], ref, rtol=1e-12, atol=1e-12)


def test_head_permutation_equivariance():
    p = problem(K=0, seed=7)
    H = p["H"]
    dh = p["y"].shape[2] // H
    perm = np.array([2, 0, 1])
    idx = (perm[:, None] * dh + np.arange(dh)[None, :]).reshape(-1)
    z = fwd(p)
    zp = fwd(p, y=p["y"][:, :, idx], gate=p["gate"][:, :, idx], Ct=p["Ct"][np.ix_(perm, perm)])
    np.testing.assert_allclose(zp, z[:, :, idx], rtol=1e-12, atol=1e-12)


def _fd(f, x, eps=1e-6):
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        xp = x.copy(); xp[i] += eps
        xm = x.copy(); xm[i] -= eps
        g[i] = (f(xp) - f(xm)) / (2 * eps)
    return g


@pytest.mark.parametrize("K", [0, 3])
def test_backward_matches_finite_differences(K):
    p = problem(B=1, L=5, H=2, dh=2, K=K, seed=11)
    loss = lambda **o: float(np.sum(p["dz"] * fwd(p, **o)))
    dy, dgate, dv, dCt, dlam, dw, ds = O.epilogue_bwd(p["y"], p["gate"], p["v"], p["dz"], p["Ct"],
                                                      p["lambda_c"], p["w"], p["s"], p["H"])
    tol = dict(rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dy, _fd(lambda a: loss(y=a), p["y"]), **tol)
    np.testing.assert_allclose(dgate, _fd(lambda a: loss(gate=a), p["gate"]), **tol)
    np.testing.assert_allclose(dCt, _fd(lambda a: loss(Ct=a), p["Ct"]), **tol)
    np.testing.assert_allclose(dlam, _fd(lambda a: loss(lambda_c=float(a)), np.array(p["lambda_c"])), **tol)
    if K:
        np.testing.assert_allclose(dv, _fd(lambda a: loss(v=a), p["v"]), **tol)
        np.testing.assert_allclose(dw, _fd(lambda a: loss(w=a), p["w"]), **tol)
        np.testing.assert_allclose(ds, _fd(lambda a: loss(s=a), p["s"]), **tol)


def test_planted_mistakes_are_caught():
    """A dropped tanh, a transposed coupling, an off-by-one tap and a wrong gate
    derivative each fail one of the pins above."""
    import oracle.epilogue_oracle as E
    p = problem(K=3, seed=13)

    def fails(patched_fwd=None, patched_bwd=None):
        keep = (E.epilogue_fwd, E.epilogue_bwd, O.epilogue_fwd, O.epilogue_bwd)
        try:
            if patched_fwd:
                E.epilogue_fwd = O.epilogue_fwd = patched_fwd
            if patched_bwd:
                E.epilogue_bwd = O.epilogue_bwd = patched_bwd
            for t in (test_coupling_against_loops, test_local_path_impulse_response,
                      lambda: test_backward_matches_finite_differences(3)):
                try:
                    t()
                except AssertionError:
                    return True
            return False
        finally:
            E.epilogue_fwd, E.epilogue_bwd, O.epilogue_fwd, O.epilogue_bwd = keep

    def no_tanh(y, gate, v, Ct, lc, w, s, H):
        return _fwd_variant(y, gate, v, Ct, lc, w, s, H, tanh=lambda a: a)

    def transposed(y, gate, v, Ct, lc, w, s, H):
        return _fwd_variant(y, gate, v, Ct, lc, w, s, H, transpose=True)

    def tap_shift(y, gate, v, Ct, lc, w, s, H):
        return _fwd_variant(y, gate, v, Ct, lc, w, s, H, shift=1)

    assert fails(patched_fwd=no_tanh)
    assert fails(patched_fwd=transposed)
    assert fails(patched_fwd=tap_shift)
    obwd = E.epilogue_bwd

    def bad_gate_grad(*a):
        r = list(obwd(*a))
        r[1] = r[1] * 2.0
        return tuple(r)
    assert fails(patched_bwd=bad_gate_grad)


def _fwd_variant(y, gate, v, Ct, lc, w, s, H, tanh=np.tanh, transpose=False, shift=0):
    """The forward with one plausible mistake planted (for the test above)."""
    y = np.asarray(y, dtype=np.float64)
    B, L, D = y.shape
    C = np.eye(H) + lc / np.sqrt(H) * tanh(np.asarray(Ct, dtype=np.float64))
    if transpose:
        C = C.T
    ybar = np.einsum("gh,blhj->blgj", C, y.reshape(B, L, H, D // H)).reshape(y.shape)
    z = expit(gate) * ybar
    K = w.shape[1]
    l = np.zeros((B, L, D))
    for k in range(K):
        kk = k + shift
        if kk < L:
            l[:, kk:, :] += w[None, None, :, k] * v[:, :L - kk, :]
    return z + s[None, None, :] * l
