"""GPU parity of the grouped linear projection and of the mixer block forward
(Sec. 3.1, 3.4) against the CPU oracle, through the C ABI.

Tolerances.  Grouped linear: float32 1e-5 (float32 products summed in float32
over at most 256 terms); bf16 inputs give exact products summed in float32 and
one bf16 rounding of the result, 1e-2.  Block: float32 1e-4 (the mixing
bound); bf16 2.5e-2: the block rounds u, g, y and z to bf16 (four roundings of
at most 2^-9 relative each, carried through maps of gain about one) and its
output once more, and the oracle rounds none of them.
"""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import act64, dev_act, dev_f32, host, rel_err, say

pytestmark = pytest.mark.gpu

ops = None


def setup_module(module):
    global ops
    from paper_2607_05583_amd import ops as _ops
    ops = _ops
    assert torch.cuda.is_available(), "GPU tests need a HIP device"


@pytest.mark.parametrize("N,G,di,dq,act", [(1, 1, 3, 5, "f32"), (1000, 4, 64, 64, "f32"), (777, 8, 32, 32, "bf16"),
                                           (4096, 1, 256, 256, "bf16"), (130, 3, 7, 11, "f32")])
def test_grouped_linear_parity(N, G, di, dq, act):
    say(f"grouped linear N={N} G={G} di={di} dq={dq} {act}")
    r = np.random.default_rng(N + G)
    x = W._act(r, (N, G * di), act)
    Wt = W._act(r, (G, di, dq), act)
    y = ops.resonator_grouped_linear(dev_act(x, act), dev_act(Wt, act))
    torch.cuda.synchronize()
    ref = O.grouped_linear(act64(x, act), act64(Wt, act))
    err = rel_err(host(y), ref)
    say(f"  err {err:.2e}")
    assert err <= (1e-5 if act == "f32" else 1e-2)


# Shapes the MFMA projection kernel takes (d_in/G a multiple of 32 for bf16 and
# 16 for float32, d_out/G a multiple of 16 up to 128, a row of at most 1 KB):
# paired and unpaired output blocks, several fragments per group, ragged and
# short token tails, the longest row.
MFMA_SHAPES = [
    (777, 8, 32, 32, "bf16"),   # the block's shape: one fragment, one pair of output blocks; ragged tail
    (5, 8, 32, 32, "bf16"),     # fewer tokens than one tile
    (1000, 4, 64, 48, "bf16"),  # two fragments per group; a pair and an unpaired block
    (333, 2, 32, 16, "bf16"),   # one unpaired block
    (513, 2, 256, 64, "bf16"),  # a 1 KB row (16 pieces per lane), 64 KB of staged weight
    (1000, 4, 64, 64, "f32"),
    (300, 16, 16, 16, "f32"),   # a 1 KB row of float32; unpaired blocks
    (257, 2, 48, 80, "f32"),    # three fragments; two pairs and an unpaired block
]


def _off_by_one(t, shape):
    """A buffer of the given shape one element into a larger allocation (aligned
    to its element, not to 16 bytes, so the projection takes the library GEMM),
    holding a copy of t when t has that shape."""
    buf = torch.empty(int(np.prod(shape)) + 1, dtype=t.dtype, device=t.device)
    v = buf[1:].view(shape)
    if tuple(t.shape) == tuple(shape):
        v.copy_(t)
    return v


@pytest.mark.parametrize("N,G,di,dq,act", MFMA_SHAPES)
def test_grouped_linear_mfma_parity(N, G, di, dq, act):
    say(f"grouped linear (MFMA kernel and library GEMM) N={N} G={G} di={di} dq={dq} {act}")
    r = np.random.default_rng(7 * N + G)
    x = W._act(r, (N, G * di), act)
    Wt = W._act(r, (G, di, dq), act)
    xd, wd = dev_act(x, act), dev_act(Wt, act)
    y = ops.resonator_grouped_linear(xd, wd)
    xo = _off_by_one(xd, tuple(xd.shape))
    yo = _off_by_one(xd, (N, G * dq))
    ops.resonator_grouped_linear(xo, wd, out=yo)
    torch.cuda.synchronize()
    ref = O.grouped_linear(act64(x, act), act64(Wt, act))
    tol = 1e-5 if act == "f32" else 1e-2
    e_mfma, e_lib = rel_err(host(y), ref), rel_err(host(yo), ref)
    say(f"  err MFMA {e_mfma:.2e}, library {e_lib:.2e}")
    assert e_mfma <= tol and e_lib <= tol


@pytest.mark.parametrize("N,G,di,dq,act", [(777, 8, 32, 32, "bf16"), (300, 4, 16, 32, "f32"),
                                           (1000, 4, 64, 48, "bf16"), (130, 3, 7, 11, "f32")])
def test_grouped_linear2_matches_two_projections(N, G, di, dq, act):
    say(f"grouped linear, two weights N={N} G={G} di={di} dq={dq} {act}")
    r = np.random.default_rng(11 * N + G)
    x = W._act(r, (N, G * di), act)
    W0 = W._act(r, (G, di, dq), act)
    W1 = W._act(r, (G, di, dq), act)
    xd, w0, w1 = dev_act(x, act), dev_act(W0, act), dev_act(W1, act)
    y0, y1 = ops.resonator_grouped_linear2(xd, w0, w1)
    s0 = ops.resonator_grouped_linear(xd, w0)
    s1 = ops.resonator_grouped_linear(xd, w1)
    torch.cuda.synchronize()
    # the same arithmetic per output as one projection at a time
    assert torch.equal(y0, s0) and torch.equal(y1, s1)
    tol = 1e-5 if act == "f32" else 1e-2
    for yy, Wk in ((y0, W0), (y1, W1)):
        assert rel_err(host(yy), O.grouped_linear(act64(x, act), act64(Wk, act))) <= tol


@pytest.mark.parametrize("B,L,d,H,K,G,M,act", [(2, 300, 64, 4, 3, 4, 4, "f32"), (1, 1000, 256, 8, 4, 8, 8, "bf16"),
                                               (2, 257, 32, 2, 0, 1, 3, "bf16")])
def test_block_fwd_parity(B, L, d, H, K, G, M, act):
    say(f"block fwd B={B} L={L} d={d} H={H} K={K} G={G} M={M} {act}")
    p = W.block_inputs(B * L + d, B, L, d, H, K, G, M, act)
    dev = lambda a: dev_act(a, act)
    pk = ("gamma", "omega", "amp", "phase")
    o = ops.resonator_block_fwd(dev(p["x"]), dev(p["Wu"]), dev(p["Wg"]), dev(p["Wo"]), *[dev_f32(p[k]) for k in pk],
                                dev_f32(p["Ct"]), p["lambda_c"], dev_f32(p["w"]) if K else None,
                                dev_f32(p["s"]) if K else None, H)
    torch.cuda.synchronize()
    ref = O.block_fwd(act64(p["x"], act), act64(p["Wu"], act), act64(p["Wg"], act), act64(p["Wo"], act),
                      *[p[k] for k in pk], p["Ct"], p["lambda_c"], p["w"] if K else np.zeros((d, 0)), p["s"], H)
    err = rel_err(host(o), ref)
    say(f"  err {err:.2e}")
    assert err <= (1e-4 if act == "f32" else 2.5e-2)
    # the dense block-diagonal route gives the same result
    dense = tuple(ops.resonator_block_diag_weight(dev(p[k])) for k in ("Wu", "Wg", "Wo"))
    od = ops.resonator_block_fwd(dev(p["x"]), dev(p["Wu"]), dev(p["Wg"]), dev(p["Wo"]),
                                 *[dev_f32(p[k]) for k in pk], dev_f32(p["Ct"]), p["lambda_c"],
                                 dev_f32(p["w"]) if K else None, dev_f32(p["s"]) if K else None, H, dense=dense)
    torch.cuda.synchronize()
    assert rel_err(host(od), ref) <= (1e-4 if act == "f32" else 2.5e-2)


@pytest.mark.parametrize("G,di,dq,act", [(8, 32, 32, "bf16"), (3, 5, 7, "f32"), (1, 4, 4, "f32")])
def test_block_diag_weight(G, di, dq, act):
    r = np.random.default_rng(G)
    Wt = W._act(r, (G, di, dq), act)
    Wd = host(ops.resonator_block_diag_weight(dev_act(Wt, act)))[0]
    ref = np.zeros((G * di, G * dq))
    for g in range(G):
        ref[g * di:(g + 1) * di, g * dq:(g + 1) * dq] = act64(Wt, act)[g]
    assert np.array_equal(Wd, ref)


@pytest.mark.parametrize("N,G,di,dq,act", [(1000, 4, 16, 8, "f32"), (777, 8, 32, 32, "bf16"), (300, 1, 24, 40, "f32")])
def test_grouped_linear_backward_parity(N, G, di, dq, act):
    say(f"grouped linear bwd N={N} G={G} di={di} dq={dq} {act}")
    r = np.random.default_rng(N + 3 * G)
    x = W._act(r, (N, G * di), act)
    Wt = W._act(r, (G, di, dq), act)
    dy = W._act(r, (N, G * dq), act)
    dx, dW = ops.resonator_grouped_linear_bwd(dev_act(x, act), dev_act(Wt, act), dev_act(dy, act))
    # accumulation adds a second gradient of the same size
    dx2, dW2 = ops.resonator_grouped_linear_bwd(dev_act(x, act), dev_act(Wt, act), dev_act(dy, act), dx=dx.clone(),
                                                dW=dW.clone(), accumulate=True)
    torch.cuda.synchronize()
    rdx, rdW = O.grouped_linear_bwd(act64(x, act), act64(Wt, act), act64(dy, act))
    b = 1e-5 if act == "f32" else 1e-2
    assert rel_err(host(dx), rdx) <= b and rel_err(host(dW), rdW) <= 1e-5
    assert rel_err(host(dx2), 2 * rdx) <= b and rel_err(host(dW2), 2 * rdW) <= 1e-5


# Data gradients summed over n uses of one input, shapes the MFMA kernel takes
# (d_out/G a multiple of 32 for bf16 and 16 for float32, d_in/G a multiple of 16
# up to 128): the block's shape with its three gradients, paired and unpaired
# output blocks, several fragments per group, a 512-byte bf16 row (16 pieces per
# lane), ragged and short token tails.
DGRAD_SHAPES = [
    (777, 8, 32, 32, "bf16", 3),
    (777, 8, 32, 32, "bf16", 1),
    (5, 8, 32, 32, "bf16", 2),
    (1000, 4, 48, 64, "bf16", 2),   # two fragments per group; a pair and an unpaired output block
    (513, 2, 64, 256, "bf16", 1),   # 16 pieces per lane, 64 KB of staged weight
    (1000, 4, 64, 32, "f32", 2),
    (300, 16, 16, 16, "f32", 1),    # 16 pieces per lane; unpaired output blocks
    (257, 2, 80, 48, "f32", 2),     # three fragments; two pairs and an unpaired block
]


@pytest.mark.parametrize("N,G,di,dq,act,n", DGRAD_SHAPES)
def test_grouped_dgrad_sum_parity(N, G, di, dq, act, n):
    say(f"grouped data gradient, {n} inputs (MFMA kernel and library GEMM) N={N} G={G} di={di} dq={dq} {act}")
    tdt = torch.bfloat16 if act == "bf16" else torch.float32
    assert ops.grouped_dgrad_supported(n, G * di, G * dq, G, tdt)
    r = np.random.default_rng(13 * N + G + n)
    dys = [W._act(r, (N, G * dq), act) for _ in range(n)]
    Ws = [W._act(r, (G, di, dq), act) for _ in range(n)]
    dd, wd = [dev_act(a, act) for a in dys], [dev_act(a, act) for a in Ws]
    dx = ops.resonator_grouped_linear_bwd_data_sum(dd, wd)
    # accumulation onto a present dx, and the library GEMMs on unaligned views
    dx2 = ops.resonator_grouped_linear_bwd_data_sum(dd, wd, dx=dx.clone(), accumulate=True)
    do_ = [_off_by_one(a, tuple(a.shape)) for a in dd]
    dxo = _off_by_one(dd[0], (N, G * di))
    ops.resonator_grouped_linear_bwd_data_sum(do_, wd, dx=dxo)
    torch.cuda.synchronize()
    zx = np.zeros((N, G * di))
    ref = sum(O.grouped_linear_bwd(zx, act64(Wk, act), act64(dk, act))[0] for dk, Wk in zip(dys, Ws))
    # the kernel rounds the sum once; the library route adds one GEMM at a time
    # into dx and so rounds the running sum n times (bf16)
    tol = 1e-5 if act == "f32" else 1e-2
    e, e2, eo = rel_err(host(dx), ref), rel_err(host(dx2), 2 * host(dx).astype(np.float64)), rel_err(host(dxo), ref)
    say(f"  err MFMA {e:.2e}, accumulated {e2:.2e}, library {eo:.2e}")
    assert e <= tol and e2 <= tol and eo <= tol * n
    if n == 1:  # the one-gradient entry point is the same kernel
        d1, _ = ops.resonator_grouped_linear_bwd(None, wd[0], dd[0])
        torch.cuda.synchronize()
        assert torch.equal(d1, dx)


# Weight gradients summed over n gradients into one or two weights, shapes the
# MFMA kernel takes (bf16; d_in, d_out multiples of 64 up to 256; d_in/G, d_out/G
# multiples of 16; at most 64 output blocks): the block's drive and gate weights
# from its three gradients, at a ragged length and at the full B4 L32K token
# count; work-groups with partial and empty token ranges; one output block per
# group; a single group.
WGRAD_SHAPES = [
    (777, 8, 32, 32, (0, 0, 1)),
    (131072, 8, 32, 32, (0, 0, 1)),
    (5, 8, 32, 32, (0,)),
    (40000, 4, 64, 16, (0, 1)),
    (33, 1, 64, 128, (1, 0)),
    (1000, 2, 64, 96, (0,)),
]


@pytest.mark.parametrize("N,G,di,dq,outs", WGRAD_SHAPES)
def test_grouped_wgrad_sum_parity(N, G, di, dq, outs):
    n, nout = len(outs), max(outs) + 1
    say(f"grouped weight gradient, {n} gradients into {nout} weights N={N} G={G} di={di} dq={dq} bf16")
    assert ops.grouped_wgrad_supported(n, nout, G * di, G * dq, G, torch.bfloat16)
    r = np.random.default_rng(17 * N + G + n)
    x = W._act(r, (N, G * di), "bf16")
    dys = [W._act(r, (N, G * dq), "bf16") for _ in range(n)]
    xd, dd = dev_act(x, "bf16"), [dev_act(a, "bf16") for a in dys]
    mk = lambda: [torch.empty((G, di, dq), dtype=torch.float32, device=xd.device) for _ in range(nout)]
    dW = ops.resonator_grouped_linear_bwd_weight_sum(xd, dd, list(outs), mk())
    dW_again = ops.resonator_grouped_linear_bwd_weight_sum(xd, dd, list(outs), mk())
    dW_acc = ops.resonator_grouped_linear_bwd_weight_sum(xd, dd, list(outs), [t.clone() for t in dW], accumulate=True)
    # the library GEMMs (one per gradient) on unaligned views of the same data
    xo = _off_by_one(xd, tuple(xd.shape))
    dW_lib = ops.resonator_grouped_linear_bwd_weight_sum(xo, [_off_by_one(a, tuple(a.shape)) for a in dd], list(outs),
                                                         mk())
    torch.cuda.synchronize()
    x64 = act64(x, "bf16")
    zW = np.zeros((G, di, dq))
    for m in range(nout):
        ref = sum(O.grouped_linear_bwd(x64, zW, act64(dk, "bf16"))[1] for dk, o in zip(dys, outs) if o == m)
        e, ea, el = rel_err(host(dW[m]), ref), rel_err(host(dW_acc[m]), 2 * ref), rel_err(host(dW_lib[m]), ref)
        say(f"  weight {m}: err MFMA {e:.2e}, accumulated {ea:.2e}, library {el:.2e}")
        assert e <= 1e-5 and ea <= 1e-5 and el <= 1e-5
        assert torch.equal(dW[m], dW_again[m])  # fixed summation order


@pytest.mark.parametrize("B,L,d,H,K,G,M,act", [(2, 300, 64, 4, 3, 4, 4, "f32"), (1, 1000, 256, 8, 4, 8, 8, "bf16"),
                                               (2, 257, 32, 2, 0, 1, 3, "f32")])
def test_block_bwd_parity(B, L, d, H, K, G, M, act):
    say(f"block bwd B={B} L={L} d={d} H={H} K={K} G={G} M={M} {act}")
    p = W.block_inputs(7 * B * L + d, B, L, d, H, K, G, M, act)
    r = np.random.default_rng(d)
    do = W._act(r, (B, L, d), act)
    dev = lambda a: dev_act(a, act)
    pk = ("gamma", "omega", "amp", "phase")
    args = [dev(p["x"]), dev(p["Wu"]), dev(p["Wg"]), dev(p["Wo"]), *[dev_f32(p[k]) for k in pk], dev_f32(p["Ct"]),
            p["lambda_c"], dev_f32(p["w"]) if K else None, dev_f32(p["s"]) if K else None, H, dev(do)]
    gr = ops.resonator_block_bwd(*args)
    dense = tuple(ops.resonator_block_diag_weight(dev(p[k])) for k in ("Wu", "Wg", "Wo"))
    grd = ops.resonator_block_bwd(*args, dense=dense)
    # the forward's saved intermediates instead of the recomputation: the same
    # kernels produced them, so the gradients are bitwise the recomputed ones
    out, saved = ops.resonator_block_fwd(*args[:-1], save=True)
    grs = ops.resonator_block_bwd(*args, saved=saved)
    out_plain = ops.resonator_block_fwd(*args[:-1])
    torch.cuda.synchronize()
    assert torch.equal(out, out_plain)
    for k, v in gr.items():
        assert (v is None and grs[k] is None) or torch.equal(v, grs[k]), k
    ref = O.block_bwd(act64(p["x"], act), act64(p["Wu"], act), act64(p["Wg"], act), act64(p["Wo"], act),
                      *[p[k] for k in pk], p["Ct"], p["lambda_c"], p["w"] if K else np.zeros((d, 0)), p["s"], H,
                      act64(do, act))
    # bf16: the backward rounds the recomputed u, g, y, z and the gradients dz,
    # dy, dgate, dv and the mixing's dx to bf16 (about ten roundings of at most
    # 2^-9 relative, some multiplied together, as in dgate = dz ybar sg (1 - sg)),
    # none of which the oracle rounds; the float32 cases check the chain itself
    b_act, b_par = (1e-4, 1e-4) if act == "f32" else (4e-2, 4e-2)
    for g in (gr, grd):
        errs = {}
        for k, v in ref.items():
            if v is None:
                assert g[k] is None
                continue
            errs[k] = rel_err(host(g[k]).reshape(np.shape(v)), v)
        say("  errs " + " ".join(f"{k}={e:.2e}" for k, e in errs.items()))
        for k, e in errs.items():
            assert e <= (b_act if k == "dx" else b_par), k


@pytest.mark.parametrize("B,L,d,H,K,G,M,act,use_dense", [(2, 300, 64, 4, 3, 4, 4, "f32", False),
                                                         (4, 2048, 256, 8, 4, 8, 8, "bf16", True)])
def test_block_forward_graph_replays_match_eager(B, L, d, H, K, G, M, act, use_dense):
    """The captured block forward, replayed three times with new inputs (eager work
    and synchronisations between the replays), equals the eager block bitwise."""
    say(f"block forward graph B={B} L={L} d={d} {act} dense={use_dense}")
    p = W.block_inputs(7 + L, B, L, d, H, K, G, M, act)
    dev = lambda a: dev_act(a, act)
    ws = [dev(p[k]) for k in ("Wu", "Wg", "Wo")]
    prm = [dev_f32(p[k]) for k in ("gamma", "omega", "amp", "phase")]
    args = (*ws, *prm, dev_f32(p["Ct"]), p["lambda_c"], dev_f32(p["w"]), dev_f32(p["s"]), H)
    dense = tuple(ops.resonator_block_diag_weight(t) for t in ws) if use_dense else None
    x0 = dev(p["x"])
    bg = ops.BlockForwardGraph(x0, *args, dense=dense)
    for r in range(3):
        xr = (x0.float() * (1.0 + 0.25 * r)).flip(1).contiguous().to(x0.dtype)
        ref = ops.resonator_block_fwd(xr, *args, dense=dense)
        torch.cuda.synchronize()
        out = bg.replay(xr)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), r
        _ = (xr.float() * 3).sum().item()  # unrelated eager work between the replays


@pytest.mark.parametrize("G,di,dq", [(1, 5, 3), (8, 32, 32), (3, 7, 11)])
def test_block_diag_extract_inverts_block_diag_and_accumulates(G, di, dq):
    r = np.random.default_rng(G * 100 + di)
    Wt = r.normal(size=(G, di, dq)).astype(np.float32)
    Wd = ops.resonator_block_diag_weight(dev_f32(Wt))
    back = ops.resonator_block_diag_extract(Wd, G)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(back), Wt)
    # off-diagonal entries are ignored; accumulate adds
    full = r.normal(size=(G * di, G * dq)).astype(np.float32)
    out = dev_f32(Wt.copy())
    ops.resonator_block_diag_extract(dev_f32(full), G, out=out, accumulate=True)
    torch.cuda.synchronize()
    ref = Wt.copy()
    for g in range(G):
        ref[g] += full[g * di:(g + 1) * di, g * dq:(g + 1) * dq]
    np.testing.assert_array_equal(host(out), ref)


@pytest.mark.parametrize("N,G,di,dq,act", [(1, 1, 3, 5, "f32"), (1000, 4, 64, 64, "f32"), (131072, 8, 32, 32, "bf16"),
                                           (70001, 3, 7, 11, "f32")])
def test_split_weight_gradient_matches_oracle_and_unsplit(N, G, di, dq, act):
    """The split-contraction weight gradient: the oracle's grouped gradient, and
    the unsplit form to float32 summation order; accumulate adds."""
    say(f"split weight gradient N={N} G={G} di={di} dq={dq} {act}")
    r = np.random.default_rng(N + 3 * G)
    x = W._act(r, (N, G * di), act)
    dy = W._act(r, (N, G * dq), act)
    xd, dyd = dev_act(x, act), dev_act(dy, act)
    dW = torch.empty((G, di, dq), dtype=torch.float32, device=xd.device)
    ops.resonator_grouped_linear_bwd_weight_split(xd, dyd, dW)
    _, dWu = ops.resonator_grouped_linear_bwd(xd, None, dyd, dW=torch.empty_like(dW))
    dW2 = dW.clone()
    ops.resonator_grouped_linear_bwd_weight_split(xd, dyd, dW2, accumulate=True)
    torch.cuda.synchronize()
    _, ref = O.grouped_linear_bwd(act64(x, act), np.zeros((G, di, dq)), act64(dy, act))
    err = rel_err(host(dW), ref)
    say(f"  err vs oracle {err:.2e}, vs unsplit {rel_err(host(dW), host(dWu)):.2e}")
    assert err <= 1e-5 and rel_err(host(dW), host(dWu)) <= 1e-5
    assert rel_err(host(dW2), 2 * ref) <= 1e-5
