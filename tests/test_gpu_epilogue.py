"""GPU parity of the mixer epilogue (head coupling, gate, local path; Sec. 3.4)
against the CPU oracle, through the C ABI.

Tolerances: float32 activations 1e-4 (sigmoid and tanh in float32, sums in
float32); bf16 activations 1.5e-2 for the outputs (one bf16 rounding of the
result, 2^-8 relative, plus float32 arithmetic on exact bf16 inputs) and 1e-3
for the parameter gradients (float32 partial sums of exact products, float64
across blocks).
"""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import act64, dev_act, dev_f32, host, rel_err, say

pytestmark = pytest.mark.gpu

ops = None

CASES = [
    # (B, L, H, dh, K, act): ragged L, odd dh (one channel per thread), K = 0, one head
    (2, 37, 4, 6, 3, "f32"),
    (2, 37, 4, 6, 3, "bf16"),
    (1, 70, 3, 5, 4, "f32"),
    (1, 70, 3, 5, 4, "bf16"),
    (2, 65, 8, 4, 0, "bf16"),
    (1, 40, 1, 16, 2, "f32"),
    (1, 33, 32, 2, 16, "f32"),
    # 16-byte (forward) and 8-byte (backward) channel pieces, several chunks per block
    (2, 77, 8, 32, 4, "bf16"),
    (1, 50, 4, 16, 3, "f32"),
    (1, 45, 2, 96, 2, "bf16"),   # 24 / 48 pieces a row: not a power of two
    (1, 30, 16, 8, 2, "bf16"),   # more than eight heads
    (1, 20, 4, 72, 2, "bf16"),   # D = 288
    (1, 20, 3, 91, 2, "f32"),    # D = 273, one channel per thread: the generic kernels
    (1, 6, 4, 1040, 3, "f32"),   # taps too many for LDS: read from global memory
]


def setup_module(module):
    global ops
    from paper_2607_05583_amd import ops as _ops
    ops = _ops
    assert torch.cuda.is_available(), "GPU tests need a HIP device"


def _dev_inputs(p, act):
    K = p["K"]
    t = {k: dev_act(p[k], act) for k in ("y", "gate", "v", "dz")}
    t["Ct"] = dev_f32(p["Ct"])
    t["w"] = dev_f32(p["w"]) if K else None
    t["s"] = dev_f32(p["s"]) if K else None
    return t


def _ref_inputs(p, act):
    return {k: act64(p[k], act) for k in ("y", "gate", "v", "dz")}


def _bounds(act):
    return (1e-4, 1e-4) if act == "f32" else (1.5e-2, 1e-3)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B{}_L{}_H{}_dh{}_K{}_{}".format(*c))
def test_epilogue_fwd_parity(case):
    B, L, H, dh, K, act = case
    say(f"epilogue fwd {case}")
    p = W.epilogue_inputs(7, B, L, H, dh, K, act)
    t = _dev_inputs(p, act)
    z = ops.resonator_epilogue_fwd(t["y"], t["gate"], t["v"] if K else None, t["Ct"], p["lambda_c"], t["w"],
                                   t["s"], H)
    torch.cuda.synchronize()
    r = _ref_inputs(p, act)
    ref = O.epilogue_fwd(r["y"], r["gate"], r["v"], p["Ct"], p["lambda_c"], p["w"] if K else None, p["s"], H)
    err = rel_err(host(z), ref)
    say(f"  err {err:.2e}")
    assert err <= _bounds(act)[0]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B{}_L{}_H{}_dh{}_K{}_{}".format(*c))
def test_epilogue_bwd_parity(case):
    B, L, H, dh, K, act = case
    say(f"epilogue bwd {case}")
    p = W.epilogue_inputs(8, B, L, H, dh, K, act)
    t = _dev_inputs(p, act)
    g = ops.resonator_epilogue_bwd(t["y"], t["gate"], t["v"] if K else None, t["dz"], t["Ct"], p["lambda_c"],
                                   t["w"], t["s"], H)
    torch.cuda.synchronize()
    r = _ref_inputs(p, act)
    ref = O.epilogue_bwd(r["y"], r["gate"], r["v"], r["dz"], p["Ct"], p["lambda_c"], p["w"] if K else None,
                         p["s"], H)
    names = ("dy", "dgate", "dv", "dCt", "dlambda_c", "dw", "ds")
    b_act, b_par = _bounds(act)
    errs = {}
    for i, n in enumerate(names):
        if ref[i] is None:
            assert g[i] is None
            continue
        errs[n] = rel_err(host(g[i]).reshape(np.shape(ref[i])), ref[i])
    say("  errs " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for n, e in errs.items():
        assert e <= (b_act if n in ("dy", "dgate", "dv") else b_par), n


def test_epilogue_bwd_is_deterministic():
    B, L, H, dh, K, act = 2, 300, 8, 8, 4, "bf16"
    say("epilogue bwd determinism")
    p = W.epilogue_inputs(9, B, L, H, dh, K, act)
    t = _dev_inputs(p, act)
    a = ops.resonator_epilogue_bwd(t["y"], t["gate"], t["v"], t["dz"], t["Ct"], p["lambda_c"], t["w"], t["s"], H)
    b = ops.resonator_epilogue_bwd(t["y"], t["gate"], t["v"], t["dz"], t["Ct"], p["lambda_c"], t["w"], t["s"], H)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


# (B, L, H, dh, K, dq, act): the epilogue fused with the output projection (one
# group per head): the block's shape with two batch rows and a ragged last tile;
# short rows, so that batch rows start inside a 16-row tile; rows of one and
# two steps (no earlier tap inside the row); no local path; float32 heads of 16.
FUSED = [
    (2, 300, 8, 32, 4, 32, "bf16"),
    (3, 17, 4, 32, 3, 16, "bf16"),
    (5, 1, 8, 32, 4, 32, "bf16"),
    (4, 2, 8, 32, 2, 32, "bf16"),
    (2, 45, 8, 32, 0, 32, "bf16"),
    (2, 100, 4, 16, 2, 32, "f32"),
    (1, 33, 2, 16, 4, 16, "f32"),
]


@pytest.mark.parametrize("case", FUSED, ids=lambda c: "B{}_L{}_H{}_dh{}_K{}_dq{}_{}".format(*c))
def test_epilogue_proj_fused_matches_two_calls_and_oracle(case):
    B, L, H, dh, K, dq, act = case
    say(f"epilogue + output projection fused {case}")
    p = W.epilogue_inputs(13, B, L, H, dh, K, act)
    t = _dev_inputs(p, act)
    r = np.random.default_rng(B * L + H)
    Wo = W._act(r, (H, dh, dq), act)
    Wd = dev_act(Wo, act)
    v = t["v"] if K else None
    assert ops.epilogue_proj_supported(t["y"], H, K, Wd)
    o = ops.resonator_epilogue_proj_fwd(t["y"], t["gate"], v, t["Ct"], p["lambda_c"], t["w"], t["s"], H, Wd)
    z = ops.resonator_epilogue_fwd(t["y"], t["gate"], v, t["Ct"], p["lambda_c"], t["w"], t["s"], H)
    o2 = ops.resonator_grouped_linear(z, Wd)
    zk = torch.empty_like(t["y"])
    o3 = ops.resonator_epilogue_proj_fwd(t["y"], t["gate"], v, t["Ct"], p["lambda_c"], t["w"], t["s"], H, Wd, z=zk)
    torch.cuda.synchronize()
    # the epilogue alone on the column kernel (unaligned copies of the inputs)
    def unaligned(a):
        buf = torch.empty(a.numel() + 1, dtype=a.dtype, device=a.device)
        u_ = buf[1:].view(a.shape)
        u_.copy_(a)
        return u_
    zc = unaligned(torch.zeros_like(z))
    ops.resonator_epilogue_fwd(unaligned(t["y"]), unaligned(t["gate"]), unaligned(v) if K else None, t["Ct"],
                               p["lambda_c"], t["w"], t["s"], H, out=zc)
    torch.cuda.synchronize()
    # the same arithmetic and roundings as the epilogue followed by the projection;
    # the kept z, the epilogue on the fused layout and on the column kernel agree bitwise
    assert torch.equal(o, o2) and torch.equal(o3, o) and torch.equal(zk, z) and torch.equal(zc, z)
    rr = _ref_inputs(p, act)
    zr = O.epilogue_fwd(rr["y"], rr["gate"], rr["v"], p["Ct"], p["lambda_c"], p["w"] if K else None, p["s"], H)
    ref = O.grouped_linear(zr, act64(Wo, act))
    err = rel_err(host(o), ref)
    say(f"  err {err:.2e}")
    # bf16: z and the output are each rounded once (2^-9 relative each)
    assert err <= (1e-4 if act == "f32" else 2.5e-2)


def test_epilogue_fwd_full_size_sampled():
    """The prefill shape (B4 L32768, H8 x dh32 = 256 channels, K = 4, bf16), checked
    on sampled rows against the oracle evaluated on those rows and their K-1
    predecessors."""
    B, L, H, dh, K, act = 4, 32768, 8, 32, 4, "bf16"
    say("epilogue fwd full size")
    p = W.epilogue_inputs(10, B, L, H, dh, K, act)
    t = _dev_inputs(p, act)
    z = ops.resonator_epilogue_fwd(t["y"], t["gate"], t["v"], t["Ct"], p["lambda_c"], t["w"], t["s"], H)
    torch.cuda.synchronize()
    zh = host(z)
    rng = np.random.default_rng(0)
    for b, t0 in zip(rng.integers(0, B, 12), rng.integers(0, L, 12)):
        lo = max(0, t0 - (K - 1))
        sl = lambda a: act64(a[b:b + 1, lo:t0 + 1], act)
        ref = O.epilogue_fwd(sl(p["y"]), sl(p["gate"]), sl(p["v"]), p["Ct"], p["lambda_c"], p["w"], p["s"], H)
        err = rel_err(zh[b, t0], ref[0, -1])
        assert err <= 1.5e-2, (b, t0, err)


def test_epilogue_bwd_many_blocks():
    """More row chunks than backward blocks (each block loops over chunks and keeps
    its parameter sums across them): B2 L40000 H8 dh32 K4 bf16, every output."""
    B, L, H, dh, K, act = 2, 40000, 8, 32, 4, "bf16"
    say("epilogue bwd many blocks")
    p = W.epilogue_inputs(11, B, L, H, dh, K, act)
    t = _dev_inputs(p, act)
    g = ops.resonator_epilogue_bwd(t["y"], t["gate"], t["v"], t["dz"], t["Ct"], p["lambda_c"], t["w"], t["s"], H)
    torch.cuda.synchronize()
    r = _ref_inputs(p, act)
    ref = O.epilogue_bwd(r["y"], r["gate"], r["v"], r["dz"], p["Ct"], p["lambda_c"], p["w"], p["s"], H)
    names = ("dy", "dgate", "dv", "dCt", "dlambda_c", "dw", "ds")
    errs = {n: rel_err(host(g[i]).reshape(np.shape(ref[i])), ref[i]) for i, n in enumerate(names)}
    say("  errs " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for n, e in errs.items():
        assert e <= (1.5e-2 if n in ("dy", "dgate", "dv") else 1e-3), n
