"""CPU oracle for the grouped linear projections and the mixer block forward of
ResonatorLM (arXiv 2607.05583, Sec. 3.1 drive/gate projection and Sec. 3.4
output projection).

TEST INFRASTRUCTURE ONLY.  The slow, obviously correct reference for the GPU
block path.  Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import it; it imports nothing from the product path.
All arithmetic is float64.

  grouped linear   y[:, g-th output slice] = x[:, g-th input slice] @ W[g]
                   (G groups; W[g] is [d_in / G, d_out / G]; a block-diagonal
                   weight)                                            Sec. 3.1, 3.4
  block forward    u = GL(x, W_u), g = GL(x, W_g)          drive and gate, Sec. 3.1
                   y = mix(u)                              Sec. 3.2 / 3.3
                   z = sigmoid(g) * (C y) + s * conv(u)    Sec. 3.4 (epilogue oracle)
                   o = GL(z, W_out)                        Sec. 3.4 output projection

Readings (each also in the design notes): the number of groups is a free
argument (the benchmark takes one group per head); the drive and the gate come
from two projections of the block input; the local path reads the drive u.

Parity status: ``grouped_linear`` is pinned by brute-force loops and by the
equivalent dense product with the explicit block-diagonal weight; ``block_fwd``
by the same composition with the direct O(L^2) mixing form in place of the
recurrence; ``grouped_linear_bwd`` by the block-diagonal products and
``block_bwd`` by central finite differences of ``block_fwd``
(``tests/test_block_oracle.py``).
"""
from __future__ import annotations

import numpy as np

from .epilogue_oracle import epilogue_bwd, epilogue_fwd
from .resonator_oracle import mix_bwd, mix_recurrence

__all__ = ["grouped_linear", "grouped_linear_bwd", "block_fwd", "block_bwd"]


def grouped_linear(x, W):
    """x [..., d_in], W [G, d_in / G, d_out / G] -> [..., d_out]."""
    x = np.asarray(x, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    G, di, do = W.shape
    assert x.shape[-1] == G * di
    out = np.empty(x.shape[:-1] + (G * do,))
    for g in range(G):
        out[..., g * do:(g + 1) * do] = x[..., g * di:(g + 1) * di] @ W[g]
    return out


def block_fwd(x, Wu, Wg, Wo, gamma, omega, amp, phase, Ct, lambda_c, w, s, H: int, mix=None):
    """The mixer block forward: o = GL(epilogue(mix(GL(x, Wu)), GL(x, Wg), GL(x, Wu)), Wo).

    ``mix`` defaults to the recurrence form; a pin passes the direct form."""
    u = grouped_linear(x, Wu)
    g = grouped_linear(x, Wg)
    y = mix_recurrence(u, gamma, omega, amp, phase)[0] if mix is None else mix(u, gamma, omega, amp, phase)
    z = epilogue_fwd(y, g, u, Ct, lambda_c, w, s, H)
    return grouped_linear(z, Wo)


def grouped_linear_bwd(x, W, dy):
    """Gradients of sum(dy * grouped_linear(x, W)): (dx, dW), per group
    dx_g = dy_g W[g]^T and dW[g] = x_g^T dy_g summed over all leading indices."""
    x = np.asarray(x, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    G, di, do = W.shape
    xf = x.reshape(-1, G * di)
    dyf = dy.reshape(-1, G * do)
    dx = np.empty_like(xf)
    dW = np.empty_like(W)
    for g in range(G):
        dx[:, g * di:(g + 1) * di] = dyf[:, g * do:(g + 1) * do] @ W[g].T
        dW[g] = xf[:, g * di:(g + 1) * di].T @ dyf[:, g * do:(g + 1) * do]
    return dx.reshape(x.shape), dW


def block_bwd(x, Wu, Wg, Wo, gamma, omega, amp, phase, Ct, lambda_c, w, s, H: int, do):
    """Gradients of sum(do * block_fwd(...)) by the chain rule through the block's
    steps (output projection, epilogue, mixing, input projections).  Returns a
    dict with dx, dWu, dWg, dWo, dgamma, domega, damp, dphase, dCt, dlambda_c,
    dw, ds (dw, ds None when K = 0)."""
    u = grouped_linear(x, Wu)
    g = grouped_linear(x, Wg)
    y = mix_recurrence(u, gamma, omega, amp, phase)[0]
    z = epilogue_fwd(y, g, u, Ct, lambda_c, w, s, H)
    dz, dWo = grouped_linear_bwd(z, Wo, do)
    dy, dg, dv, dCt, dlam, dw, ds = epilogue_bwd(y, g, u, dz, Ct, lambda_c, w, s, H)
    mb = mix_bwd(u, dy, gamma, omega, amp, phase)
    du = mb["dx"] + (dv if dv is not None else 0.0)
    dxu, dWu = grouped_linear_bwd(x, Wu, du)
    dxg, dWg = grouped_linear_bwd(x, Wg, dg)
    return dict(dx=dxu + dxg, dWu=dWu, dWg=dWg, dWo=dWo, dgamma=mb["dgamma"], domega=mb["domega"],
                damp=mb["damp"], dphase=mb["dphase"], dCt=dCt, dlambda_c=dlam, dw=dw, ds=ds)
