"""Pins of the block oracle (grouped linear projections and the mixer block
forward; Sec. 3.1 and 3.4).

No GPU.  The grouped linear is pinned by brute-force loops over every output
element and by the dense product with the explicit block-diagonal weight; the
block forward by the same composition with the direct O(L^2) mixing form, and by
the closed form of a block whose projections are identities, whose coupling and
local path are off.  Planted mistakes (groups taken from the wrong input slice,
the gate and drive swapped) each fail a pin.
"""
import numpy as np
import pytest
from scipy.special import expit

import oracle as O
import oracle.block_oracle as BO


def _gl_loops(x, W):
    G, di, do = W.shape
    N = x.shape[0]
    out = np.zeros((N, G * do))
    for n in range(N):
        for g in range(G):
            for o in range(do):
                acc = 0.0
                for i in range(di):
                    acc += x[n, g * di + i] * W[g, i, o]
                out[n, g * do + o] = acc
    return out


def _block_diag(W):
    G, di, do = W.shape
    M = np.zeros((G * di, G * do))
    for g in range(G):
        M[g * di:(g + 1) * di, g * do:(g + 1) * do] = W[g]
    return M


@pytest.mark.parametrize("G,di,do", [(1, 3, 5), (4, 2, 3), (3, 5, 1)])
def test_grouped_linear_against_loops_and_block_diagonal(G, di, do):
    r = np.random.default_rng(G * 10 + di)
    x = r.normal(size=(7, G * di))
    W = r.normal(size=(G, di, do))
    y = BO.grouped_linear(x, W)
    np.testing.assert_allclose(y, _gl_loops(x, W), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y, x @ _block_diag(W), rtol=1e-12, atol=1e-12)
    # batched leading dimensions
    np.testing.assert_allclose(BO.grouped_linear(x.reshape(7, 1, -1), W)[:, 0], y, rtol=1e-13, atol=1e-13)


def _problem(seed=0, B=2, L=30, d=8, H=2, K=3, G=2, M=3):
    r = np.random.default_rng(seed)
    D = d
    return dict(x=r.normal(size=(B, L, d)), Wu=r.normal(size=(G, d // G, D // G)) / 2,
                Wg=r.normal(size=(G, d // G, D // G)) / 2, Wo=r.normal(size=(G, D // G, d // G)) / 2,
                gamma=r.uniform(0.01, 0.5, size=(D, M)), omega=r.uniform(0, np.pi, size=(D, M)),
                amp=r.normal(size=(D, M)) / np.sqrt(M), phase=r.uniform(0, 2 * np.pi, size=(D, M)),
                Ct=r.normal(size=(H, H)), lambda_c=0.6, w=r.normal(size=(D, K)), s=r.normal(size=D), H=H)


def test_block_recurrence_and_direct_forms_agree():
    p = _problem()
    a = BO.block_fwd(**p)
    b = BO.block_fwd(**p, mix=O.mix_direct)
    np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-10)


def test_block_with_identity_projections_and_no_coupling_or_local_path():
    """W_u = W_g = W_out = I (one group), lambda_c = 0, K = 0: o = sigmoid(x) * mix(x)."""
    p = _problem(seed=3, G=1)
    d = p["x"].shape[-1]
    eye = np.eye(d)[None]
    o = BO.block_fwd(p["x"], eye, eye, eye, p["gamma"], p["omega"], p["amp"], p["phase"], p["Ct"], 0.0,
                     np.zeros((d, 0)), p["s"], p["H"])
    y = O.mix_direct(p["x"], p["gamma"], p["omega"], p["amp"], p["phase"])
    np.testing.assert_allclose(o, expit(p["x"]) * y, rtol=1e-10, atol=1e-12)


def test_planted_mistakes_are_caught():
    keep = BO.grouped_linear

    def wrong_slices(x, W):  # every group reads the first input slice
        x = np.asarray(x, dtype=np.float64)
        G, di, do = W.shape
        return np.concatenate([x[..., :di] @ W[g] for g in range(G)], axis=-1)

    try:
        BO.grouped_linear = wrong_slices
        with pytest.raises(AssertionError):
            test_grouped_linear_against_loops_and_block_diagonal(4, 2, 3)
    finally:
        BO.grouped_linear = keep

    p = _problem(seed=5, G=1)
    d = p["x"].shape[-1]
    eye = np.eye(d)[None]
    swapped = BO.block_fwd(p["x"], eye, eye * 0.5, eye, p["gamma"], p["omega"], p["amp"], p["phase"], p["Ct"],
                           0.0, np.zeros((d, 0)), p["s"], p["H"])
    y = O.mix_direct(0.5 * p["x"], p["gamma"], p["omega"], p["amp"], p["phase"])
    # drive and gate swapped would give sigmoid(x) * mix(x / 2): must differ from the true block
    assert not np.allclose(swapped, expit(p["x"]) * y, rtol=1e-6)


def test_block_backward_by_finite_differences():
    """Every gradient of the block against central differences of block_fwd."""
    p = _problem(seed=11, B=1, L=12, d=4, H=2, K=2, G=2, M=2)
    r = np.random.default_rng(0)
    do = r.normal(size=p["x"].shape)
    g = BO.block_bwd(**p, do=do)
    names = {"x": "dx", "Wu": "dWu", "Wg": "dWg", "Wo": "dWo", "gamma": "dgamma", "omega": "domega", "amp": "damp",
             "phase": "dphase", "Ct": "dCt", "w": "dw", "s": "ds"}
    h = 1e-6
    for k, gk in names.items():
        base = np.asarray(p[k], dtype=np.float64)
        flat = base.reshape(-1)
        for i in r.choice(flat.size, size=min(4, flat.size), replace=False):
            e = np.zeros_like(flat)
            e[i] = h
            fp = np.sum(do * BO.block_fwd(**{**p, k: (flat + e).reshape(base.shape)}))
            fm = np.sum(do * BO.block_fwd(**{**p, k: (flat - e).reshape(base.shape)}))
            fd = (fp - fm) / (2 * h)
            assert abs(np.asarray(g[gk]).reshape(-1)[i] - fd) <= 1e-6 * max(1.0, abs(fd)), (k, i)
    fp = np.sum(do * BO.block_fwd(**{**p, "lambda_c": p["lambda_c"] + h}))
    fm = np.sum(do * BO.block_fwd(**{**p, "lambda_c": p["lambda_c"] - h}))
    assert abs(g["dlambda_c"] - (fp - fm) / (2 * h)) <= 1e-6 * max(1.0, abs((fp - fm) / (2 * h)))


def test_grouped_linear_backward_against_block_diagonal():
    r = np.random.default_rng(4)
    x, Wt, dy = r.normal(size=(9, 12)), r.normal(size=(3, 4, 2)), r.normal(size=(9, 6))
    dx, dW = BO.grouped_linear_bwd(x, Wt, dy)
    np.testing.assert_allclose(dx, dy @ _block_diag(Wt).T, rtol=1e-12, atol=1e-12)
    full = x.T @ dy
    for g in range(3):
        np.testing.assert_allclose(dW[g], full[g * 4:(g + 1) * 4, g * 2:(g + 1) * 2], rtol=1e-12, atol=1e-12)
