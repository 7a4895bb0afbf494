"""CPU oracle for the mixer epilogue of ResonatorLM (arXiv 2607.05583, Sec. 3.4).

TEST INFRASTRUCTURE ONLY.  The slow, obviously correct reference for the HIP
epilogue kernels.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py``'s ``cpu_baseline`` leg may import it; it imports nothing from the
product path.

All arithmetic is float64.  Arrays are [B, L, D] with D = H * dh, channel
c = h * dh + j (head h, index j within the head), matching the flattening of
the head tensor in the combine equation.

What the epilogue computes, after the resonant mixing has produced y:
  coupling matrix   C = I + (lambda_c / sqrt(H)) tanh(Ct)            (Sec. 3.4, coupling eq.)
  head mixing       ybar[b,t,g*dh+j] = sum_h C[g,h] y[b,t,h*dh+j]   (Sec. 3.4, mixing eq.)
  gate              gamma_t = sigmoid(gate_t)                        (Sec. 3.1, last paragraph)
  local path        l[b,t,c] = sum_{k<K} w[c,k] v[b,t-k,c]           (Sec. 3.4, causal depthwise conv)
                    (v is the token stream the local branch reads; zero before t = 0)
  combine           z = gamma_t * ybar + s * l                       (Sec. 3.4, combine eq.)

Readings (each also in the design notes): the depthwise convolution's tap k
multiplies the drive k steps back (tap 0 = the current step); "the token
stream" is whatever tensor the caller passes as v (in the block, the mixer's
input); K = 0 disables the local path.

Parity status: ``epilogue_fwd`` is pinned by closed forms (lambda_c = 0 and
K = 0 reduce it to sigmoid(gate) * y), an impulse response of the local path,
and head-permutation equivariance; ``epilogue_bwd`` by central finite
differences of ``epilogue_fwd`` (``tests/test_epilogue_oracle.py``).
"""
from __future__ import annotations

import numpy as np

__all__ = ["coupling_matrix", "epilogue_fwd", "epilogue_bwd"]


def _sigmoid(u):
    return 1.0 / (1.0 + np.exp(-u))


def coupling_matrix(Ct, lambda_c: float) -> np.ndarray:
    """C = I + (lambda_c / sqrt(H)) tanh(Ct), [H, H] (Sec. 3.4, coupling eq.)."""
    Ct = np.asarray(Ct, dtype=np.float64)
    H = Ct.shape[0]
    return np.eye(H) + (float(lambda_c) / np.sqrt(H)) * np.tanh(Ct)


def _heads(a, H):
    B, L, D = a.shape
    return a.reshape(B, L, H, D // H)


def _local(v, w):
    """l[b,t,c] = sum_k w[c,k] v[b,t-k,c], zero before t = 0."""
    B, L, D = v.shape
    K = w.shape[1]
    l = np.zeros((B, L, D))
    for k in range(K):
        l[:, k:, :] += w[None, None, :, k] * v[:, :L - k, :]
    return l


def epilogue_fwd(y, gate, v, Ct, lambda_c, w, s, H: int):
    """z = sigmoid(gate) * ybar + s * l  (Sec. 3.4 coupling, mixing and combine equations).

    y, gate: [B, L, D]; v: [B, L, D] or None (K = 0); Ct: [H, H]; w: [D, K]; s: [D].
    """
    y = np.asarray(y, dtype=np.float64)
    gate = np.asarray(gate, dtype=np.float64)
    C = coupling_matrix(Ct, lambda_c)
    ybar = np.einsum("gh,blhj->blgj", C, _heads(y, H)).reshape(y.shape)
    z = _sigmoid(gate) * ybar
    w = np.zeros((y.shape[2], 0)) if w is None else np.asarray(w, dtype=np.float64)
    if w.shape[1] > 0:
        z = z + np.asarray(s, dtype=np.float64)[None, None, :] * _local(np.asarray(v, dtype=np.float64), w)
    return z


def epilogue_bwd(y, gate, v, dz, Ct, lambda_c, w, s, H: int):
    """Gradients of sum(dz * z) for z = epilogue_fwd(...).

    With sg = sigmoid(gate), C = I + (lc/sqrt H) tanh(Ct), ybar = C y (per head):
      dgate = dz ybar sg (1 - sg)
      dy    = C^T (dz sg)                               (per head, per position)
      dC    = sum_{b,t,j} (dz sg)[g,j] y[h,j]  ->  dCt = dC (lc/sqrt H)(1 - tanh^2 Ct),
                                                  dlambda_c = sum dC tanh(Ct) / sqrt H
      ds[c] = sum_{b,t} dz l;   dl = dz s
      dw[c,k] = sum_{b,t} dl[b,t,c] v[b,t-k,c];   dv[b,t,c] = sum_k w[c,k] dl[b,t+k,c]
    Returns (dy, dgate, dv, dCt, dlambda_c, dw, ds); dv, dw, ds are None when K = 0.
    """
    y = np.asarray(y, dtype=np.float64)
    gate = np.asarray(gate, dtype=np.float64)
    dz = np.asarray(dz, dtype=np.float64)
    Ct = np.asarray(Ct, dtype=np.float64)
    B, L, D = y.shape
    Cm = coupling_matrix(Ct, lambda_c)
    sg = _sigmoid(gate)
    ybar = np.einsum("gh,blhj->blgj", Cm, _heads(y, H)).reshape(y.shape)
    dgate = dz * ybar * sg * (1.0 - sg)
    dyb = dz * sg
    dy = np.einsum("gh,blgj->blhj", Cm, _heads(dyb, H)).reshape(y.shape)
    dC = np.einsum("blgj,blhj->gh", _heads(dyb, H), _heads(y, H))
    th = np.tanh(Ct)
    dCt = dC * (float(lambda_c) / np.sqrt(H)) * (1.0 - th * th)
    dlam = float(np.sum(dC * th) / np.sqrt(H))
    if w is None or np.asarray(w).shape[1] == 0:
        return dy, dgate, None, dCt, dlam, None, None
    w = np.asarray(w, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    K = w.shape[1]
    l = _local(v, w)
    ds = np.sum(dz * l, axis=(0, 1))
    dl = dz * s[None, None, :]
    dw = np.zeros((D, K))
    dv = np.zeros((B, L, D))
    for k in range(K):
        dw[:, k] = np.sum(dl[:, k:, :] * v[:, :L - k, :], axis=(0, 1))
        dv[:, :L - k, :] += w[None, None, :, k] * dl[:, k:, :]
    return dy, dgate, dv, dCt, dlam, dw, ds
