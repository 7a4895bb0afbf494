"""Seeded synthetic workloads for the resonant mixing operator.

This module only draws random numbers and converts float32 to bfloat16 bit
patterns; it holds none of the operator's arithmetic.  Both the CPU oracle side
(tests, bench's CPU baseline) and the HIP side (tests, bench, smoke) take their
inputs from here, so the two consume identical values.

Shapes and distributions stand in for the paper's workload: mixer drives of a
d_model = 256 character language model at 1K-32K tokens (Sec. 4; block benchmark
of Sec. 5.3).  No dataset content is used: drives are N(0, 1), the scale of the
RMS-normalised activations that feed the mixer.

Recipe (numpy PCG64, ``np.random.default_rng(seed)``):
  draw order x, gamma, omega, phi, a, then dy (training) or per-step drives
  (decode); x and dy are float32 standard normals; gamma uniform or
  log-uniform (exp of a uniform in log space); omega ~ U[0, pi];
  phi ~ U[0, 2 pi); a ~ N(0, 1/M) (variance 1/M).  bfloat16 tensors are
  round-to-nearest-even conversions of those float32 draws.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


# --------------------------------------------------------------------------
# bfloat16 conversion (bit manipulation only)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(a) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float32 (exact)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32)


# --------------------------------------------------------------------------
# parameter draws
# --------------------------------------------------------------------------
def draw_params(rng, D: int, M: int, gamma_range, gamma_log: bool):
    """Draw (gamma, omega, phase, amp) float32 [D, M] in that order."""
    lo, hi = gamma_range
    if gamma_log:
        gamma = np.exp(rng.uniform(math.log(lo), math.log(hi), size=(D, M)))
    else:
        gamma = rng.uniform(lo, hi, size=(D, M))
    omega = rng.uniform(0.0, math.pi, size=(D, M))
    phase = rng.uniform(0.0, 2.0 * math.pi, size=(D, M))
    amp = rng.normal(0.0, math.sqrt(1.0 / M), size=(D, M))
    f = lambda v: np.ascontiguousarray(v, dtype=np.float32)
    return {"gamma": f(gamma), "omega": f(omega), "phase": f(phase), "amp": f(amp)}


@dataclass(frozen=True)
class Config:
    index: int
    name: str
    kind: str             # "fwd", "decode", "train"
    B: int
    L: int
    D: int
    M: int
    act: str              # activation dtype: "f32" or "bf16"
    out: str              # output dtype
    seed: int
    gamma_range: tuple
    gamma_log: bool
    steps: int = 0        # decode steps
    layers: int = 1       # training stack depth


CONFIGS = {
    1: Config(1, "fwd_f32_B1_L1024_D64_M4", "fwd", 1, 1024, 64, 4, "f32", "f32",
              0, (1e-3, 0.5), False),
    2: Config(2, "fwd_f32_B8_L8192_D256_M8", "fwd", 8, 8192, 256, 8, "f32", "f32",
              1, (1e-4, 1.0), True),
    3: Config(3, "prefill_bf16_B4_L32768_D256_M8", "fwd", 4, 32768, 256, 8, "bf16", "bf16",
              2, (1e-5, 1.0), True),
    4: Config(4, "decode_bf16_B64_D256_M8_prompt1024_steps32768", "decode", 64, 1024, 256, 8,
              "bf16", "bf16", 3, (1e-4, 1.0), True, steps=32768),
    5: Config(5, "train_bf16_6x_B8_L8192_D256_M8", "train", 8, 8192, 256, 8, "bf16", "bf16",
              4, (1e-4, 1.0), True, layers=6),
}


def _act(rng, shape, act):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    return f32_to_bf16_bits(x) if act == "bf16" else x


def fwd_inputs(cfg: Config, B=None, L=None, D=None):
    """Inputs of a forward config: x ([B,L,D] float32 or bf16 bits) and params.

    B/L/D overrides give reduced shapes drawn with the same recipe and seed.
    """
    B = cfg.B if B is None else B
    L = cfg.L if L is None else L
    D = cfg.D if D is None else D
    rng = np.random.default_rng(cfg.seed)
    x = _act(rng, (B, L, D), cfg.act)
    p = draw_params(rng, D, cfg.M, cfg.gamma_range, cfg.gamma_log)
    return {"x": x, **p}


class DecodeInputs:
    """Decode config: prompt, params, then a stream of per-step drives.

    ``prompt`` [B, L, D] and the parameters are drawn first; ``steps(n)`` then
    returns the next n per-step drives [n, B, D] from the same generator, so the
    concatenation of successive calls is the fixed sequence of the config.
    """

    def __init__(self, cfg: Config, B=None, L=None, D=None):
        self.cfg = cfg
        self.B = cfg.B if B is None else B
        self.L = cfg.L if L is None else L
        self.D = cfg.D if D is None else D
        self._rng = np.random.default_rng(cfg.seed)
        self.prompt = _act(self._rng, (self.B, self.L, self.D), cfg.act)
        self.params = draw_params(self._rng, self.D, cfg.M, cfg.gamma_range, cfg.gamma_log)
        self.drawn = 0

    def steps(self, n: int):
        xs = _act(self._rng, (n, self.B, self.D), self.cfg.act)
        self.drawn += n
        return xs


def train_layer_inputs(cfg: Config, layer: int, B=None, L=None, D=None):
    """One layer of the training config: x, params, dy (bf16 bits or float32).

    Each layer has its own generator, seeded with the sequence (seed, layer), so a
    layer can be drawn without drawing the layers before it.  Draw order x, gamma,
    omega, phi, a, dy.
    """
    B = cfg.B if B is None else B
    L = cfg.L if L is None else L
    D = cfg.D if D is None else D
    rng = np.random.default_rng(np.random.SeedSequence([cfg.seed, layer]))
    x = _act(rng, (B, L, D), cfg.act)
    p = draw_params(rng, D, cfg.M, cfg.gamma_range, cfg.gamma_log)
    dy = _act(rng, (B, L, D), cfg.act)
    return {"x": x, "dy": dy, **p}


def random_problem(seed: int, B: int, L: int, D: int, M: int, act: str = "f32",
                   gamma_range=(1e-3, 0.5), gamma_log=False, with_h0=False, with_dy=False):
    """Small seeded problem for tests (same recipe; optional h0 and dy)."""
    rng = np.random.default_rng(seed)
    x = _act(rng, (B, L, D), act)
    p = draw_params(rng, D, M, gamma_range, gamma_log)
    out = {"x": x, **p}
    if with_h0:
        out["h0"] = rng.standard_normal(size=(B, D, M, 2), dtype=np.float32)
    if with_dy:
        out["dy"] = _act(rng, (B, L, D), act)
    return out


def act_to_f32(a, act: str) -> np.ndarray:
    """Activation array (float32 or bf16 bits) as float32 values."""
    return bf16_bits_to_f32(a) if act == "bf16" else np.asarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# mixer epilogue (head coupling, gate, local path)
# --------------------------------------------------------------------------
def epilogue_inputs(seed: int, B: int, L: int, H: int, dh: int, K: int, act: str = "f32",
                    lambda_c: float = 0.5):
    """Seeded inputs of the mixer epilogue: y, gate, v, dz [B, L, H dh] standard
    normals (float32 or bf16 bits); Ct [H, H] standard normal; w [D, K] N(0, 1/K)
    (a K-tap filter of unit gain on average); s [D] N(0, 1).  Draw order y, gate,
    v, dz, Ct, w, s."""
    rng = np.random.default_rng(seed)
    D = H * dh
    y = _act(rng, (B, L, D), act)
    gate = _act(rng, (B, L, D), act)
    v = _act(rng, (B, L, D), act)
    dz = _act(rng, (B, L, D), act)
    Ct = rng.standard_normal((H, H)).astype(np.float32)
    w = (rng.standard_normal((D, K)) / math.sqrt(max(K, 1))).astype(np.float32)
    s = rng.standard_normal(D).astype(np.float32)
    return dict(y=y, gate=gate, v=v, dz=dz, Ct=Ct, w=w, s=s, lambda_c=float(lambda_c), H=H, K=K)


# --------------------------------------------------------------------------
# mixer block (grouped projections around the mixing and the epilogue)
# --------------------------------------------------------------------------
def block_inputs(seed: int, B: int, L: int, d: int, H: int, K: int, G: int, M: int, act: str = "f32"):
    """Seeded inputs of the mixer block: x [B, L, d] standard normal; W_u, W_g,
    W_out [G, d/G, d/G] normal with variance G/d (unit gain on average); mode
    parameters as the 8K config (gamma log-uniform in [1e-4, 1]); Ct [H, H]
    standard normal, lambda_c = 0.5, taps w [d, K] N(0, 1/K), scales s [d] N(0, 1).
    Activations and weights are float32 or bf16 bits.  Draw order x, W_u, W_g,
    W_out, mode parameters, Ct, w, s."""
    rng = np.random.default_rng(seed)
    x = _act(rng, (B, L, d), act)
    sd = 1.0 / math.sqrt(d // G)
    Ws = []
    for _ in range(3):
        w32 = (rng.standard_normal((G, d // G, d // G)) * sd).astype(np.float32)
        Ws.append(f32_to_bf16_bits(w32) if act == "bf16" else w32)
    p = draw_params(rng, d, M, (1e-4, 1.0), True)
    Ct = rng.standard_normal((H, H)).astype(np.float32)
    w = (rng.standard_normal((d, K)) / math.sqrt(max(K, 1))).astype(np.float32)
    s = rng.standard_normal(d).astype(np.float32)
    return dict(x=x, Wu=Ws[0], Wg=Ws[1], Wo=Ws[2], **p, Ct=Ct, lambda_c=0.5, w=w, s=s, H=H, K=K, G=G)
