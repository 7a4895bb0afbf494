"""GPU parity of the forward path and the prompt state against the CPU oracle.

Every case compares the HIP path (through the C ABI) with the float64 oracle on
identical seeded inputs, element by element, with the error metric of
gpu_util.rel_err: 1e-4 for float32 activations, 2e-2 when bf16 is involved.
"""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import act64, dev_act, dev_f32, host, params_dev, params_np, rel_err, say, tol

pytestmark = pytest.mark.gpu

ops = None


def setup_module(module):
    global ops
    from paper_2607_05583_amd import ops as _ops
    ops = _ops
    assert torch.cuda.is_available(), "GPU tests need a HIP device"


SMALL = [
    # B, L, D, M, h0, seed
    (1, 1, 1, 1, False, 1),
    (2, 15, 3, 2, True, 2),
    (1, 16, 33, 4, False, 3),
    (2, 257, 40, 8, True, 4),
    (1, 1000, 64, 9, False, 5),
    (3, 600, 70, 16, True, 6),
    (2, 513, 32, 5, False, 7),
    (1, 2048, 96, 8, True, 8),
]


@pytest.mark.parametrize("B,L,D,M,use_h0,seed", SMALL)
@pytest.mark.parametrize("act,out", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")])
def test_fwd_small_shapes(B, L, D, M, use_h0, seed, act, out):
    say(f"fwd small B={B} L={L} D={D} M={M} h0={use_h0} {act}->{out}")
    prob = W.random_problem(seed, B, L, D, M, act=act, gamma_range=(1e-4, 1.0), gamma_log=True,
                            with_h0=use_h0)
    x = dev_act(prob["x"], act)
    h0 = dev_f32(prob["h0"]) if use_h0 else None
    y, hout = ops.resonator_mix_fwd(x, *params_dev(prob), h0=h0,
                                    out_dtype=torch.float32 if out == "f32" else x.dtype,
                                    return_state=True)
    torch.cuda.synchronize()
    yr, hr = O.mix_recurrence(act64(prob["x"], act), *params_np(prob),
                              h0=prob["h0"] if use_h0 else None)
    assert rel_err(host(y), yr) <= tol(act, out)
    assert rel_err(host(hout), hr) <= (1e-4 if act == "f32" else 2e-2)


def test_config1_against_direct_sum():
    cfg = W.CONFIGS[1]
    say(f"config 1 {cfg.name}")
    inp = W.fwd_inputs(cfg)
    x = dev_act(inp["x"], cfg.act)
    y = ops.resonator_mix_fwd(x, *params_dev(inp))
    torch.cuda.synchronize()
    yd = O.mix_direct(act64(inp["x"], cfg.act), *params_np(inp))
    e = rel_err(host(y), yd)
    say(f"config 1 rel err {e:.3e}")
    assert e <= 1e-4


def _spot_positions(rng, B, L, D, n):
    b = rng.integers(0, B, n)
    t = np.concatenate([rng.integers(0, L, n - 8), [0, 1, L - 1, L - 2, 255, 256, L // 2, L - 257]])
    d = rng.integers(0, D, n)
    return np.stack([b, t, d], 1)


@pytest.mark.parametrize("k", [2, 3])
def test_config_full_size(k):
    cfg = W.CONFIGS[k]
    say(f"config {k} {cfg.name}")
    inp = W.fwd_inputs(cfg)
    x = dev_act(inp["x"], cfg.act)
    y, hout = ops.resonator_mix_fwd(x, *params_dev(inp), return_state=True)
    torch.cuda.synchronize()
    yg, hg = host(y), host(hout)
    x64 = act64(inp["x"], cfg.act)
    yr, hr = O.mix_recurrence(x64, *params_np(inp))
    e, eh = rel_err(yg, yr), rel_err(hg, hr)
    say(f"config {k} rel err y {e:.3e} h_out {eh:.3e}")
    assert e <= tol(cfg.act, cfg.out)
    assert eh <= (1e-4 if cfg.act == "f32" else 2e-2)
    # independent direct-sum spot checks at sampled positions
    pos = _spot_positions(np.random.default_rng(100 + k), cfg.B, cfg.L, cfg.D, 96)
    yd = O.mix_direct_at(x64, *params_np(inp), pos)
    got = yg[pos[:, 0], pos[:, 1], pos[:, 2]]
    den = np.maximum(np.abs(yd), np.sqrt(np.mean(yr ** 2)))
    assert float((np.abs(got - yd) / den).max()) <= tol(cfg.act, cfg.out)


@pytest.mark.parametrize("B,L,D,M,seed", [(1, 1, 1, 1, 1), (2, 0, 5, 3, 2), (2, 255, 33, 8, 3),
                                          (3, 700, 64, 12, 4), (64, 1024, 256, 8, 5)])
@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_state_init(B, L, D, M, seed, act):
    say(f"state_init B={B} L={L} D={D} M={M} {act}")
    prob = W.random_problem(seed, B, L, D, M, act=act, gamma_range=(1e-4, 1.0), gamma_log=True)
    x = dev_act(prob["x"], act)
    st = ops.resonator_state_init(x, *params_dev(prob))
    torch.cuda.synchronize()
    ref = O.state_init(act64(prob["x"], act), *params_np(prob))
    if L == 0:
        assert np.array_equal(host(st), np.zeros_like(ref))
    else:
        assert rel_err(host(st), ref) <= (1e-4 if act == "f32" else 2e-2)


def test_causality_bitwise():
    """Sec. 3.5 causality check: perturbing the suffix leaves every earlier output bit-identical."""
    say("causality bitwise")
    prob = W.random_problem(21, 2, 3000, 64, 8, act="bf16", gamma_range=(1e-5, 1.0), gamma_log=True)
    x = dev_act(prob["x"], "bf16")
    pr = params_dev(prob)
    y1 = ops.resonator_mix_fwd(x, *pr)
    for cut in (1, 255, 256, 1500, 2999):
        x2 = x.clone()
        x2[:, cut:] = torch.randn_like(x2[:, cut:].float()).to(x2.dtype)
        y2 = ops.resonator_mix_fwd(x2, *pr)
        torch.cuda.synchronize()
        assert torch.equal(y1[:, :cut], y2[:, :cut])
        assert not torch.equal(y1[:, cut:], y2[:, cut:])


def test_split_prefill_matches_full():
    """fwd(x[:L0]) -> h_out, fwd(x[L0:], h0=h_out) reproduces fwd(x) (state hand-over)."""
    say("split prefill")
    prob = W.random_problem(22, 2, 1200, 40, 8, act="f32", gamma_range=(1e-4, 1.0), gamma_log=True)
    x = dev_act(prob["x"], "f32")
    pr = params_dev(prob)
    y, h = ops.resonator_mix_fwd(x, *pr, return_state=True)
    y1, h1 = ops.resonator_mix_fwd(x[:, :500].contiguous(), *pr, return_state=True)
    y2, h2 = ops.resonator_mix_fwd(x[:, 500:].contiguous(), *pr, h0=h1, return_state=True)
    torch.cuda.synchronize()
    yr = O.mix_recurrence(prob["x"].astype(np.float64), *params_np(prob))[0]
    assert rel_err(np.concatenate([host(y1), host(y2)], 1), yr) <= 1e-4
    assert rel_err(host(h2), host(h)) <= 1e-4


def test_fwd_repeatable():
    say("fwd repeatable")
    prob = W.random_problem(23, 2, 2000, 64, 8, act="bf16", gamma_range=(1e-5, 1.0), gamma_log=True)
    x = dev_act(prob["x"], "bf16")
    pr = params_dev(prob)
    a = ops.resonator_mix_fwd(x, *pr)
    b = ops.resonator_mix_fwd(x, *pr)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# Geometries that reach every branch of the forward's work split: many carry
# fold blocks per row, long float32 rows with an initial state, a partial last
# tile inside a multi-tile work unit, short last units, ragged channel blocks,
# units of two and three tiles.  Each is compared element by element with the
# oracle recurrence (y and h_out) and spot-checked against the direct sum.
TILING = [
    # B, L, D, M, act, out, h0, seed
    (1, 16384, 64, 8, "bf16", "bf16", False, 31),
    (1, 32768, 256, 8, "f32", "f32", True, 32),
    (4, 32001, 256, 8, "bf16", "bf16", True, 33),
    (8, 8191, 200, 8, "f32", "f32", False, 34),
    (4, 8492, 256, 8, "bf16", "bf16", True, 35),
    (4, 8192, 256, 8, "bf16", "f32", False, 36),
    (2, 5000, 96, 5, "f32", "f32", True, 37),
    (3, 4097, 130, 8, "bf16", "bf16", True, 38),
    # many chains, few work-groups each (2, 3 and 4 on 256 compute units)
    (16, 2085, 256, 8, "f32", "f32", True, 39),
    (8, 3001, 320, 8, "f32", "f32", False, 40),
    (16, 3000, 256, 8, "bf16", "bf16", True, 44),
]


@pytest.mark.parametrize("B,L,D,M,act,out,use_h0,seed", TILING)
def test_fwd_tiling_geometries(B, L, D, M, act, out, use_h0, seed):
    say(f"fwd tiling B={B} L={L} D={D} M={M} {act}->{out} h0={use_h0}")
    prob = W.random_problem(seed, B, L, D, M, act=act, gamma_range=(1e-5, 1.0), gamma_log=True,
                            with_h0=use_h0)
    x = dev_act(prob["x"], act)
    h0 = dev_f32(prob["h0"]) if use_h0 else None
    y, hout = ops.resonator_mix_fwd(x, *params_dev(prob), h0=h0,
                                    out_dtype=torch.float32 if out == "f32" else x.dtype,
                                    return_state=True)
    torch.cuda.synchronize()
    yg, hg = host(y), host(hout)
    x64 = act64(prob["x"], act)
    yr, hr = O.mix_recurrence(x64, *params_np(prob), h0=prob["h0"] if use_h0 else None)
    e, eh = rel_err(yg, yr), rel_err(hg, hr)
    say(f"  rel err y {e:.3e} h_out {eh:.3e}")
    assert e <= tol(act, out)
    assert eh <= (1e-4 if act == "f32" else 2e-2)
    pos = _spot_positions(np.random.default_rng(seed), B, L, D, 64)
    yd = O.mix_direct_at(x64, *params_np(prob), pos, h0=prob["h0"] if use_h0 else None)
    got = yg[pos[:, 0], pos[:, 1], pos[:, 2]]
    den = np.maximum(np.abs(yd), np.sqrt(np.mean(yr ** 2)))
    assert float((np.abs(got - yd) / den).max()) <= tol(act, out)


def test_h_out_may_alias_h0():
    """h_out written over h0 (in-place state hand-over) gives the same y and state
    as separate buffers, for the single-kernel forward and the M > 8 path."""
    for M, act, seed in ((8, "bf16", 41), (8, "f32", 42), (12, "f32", 43)):
        say(f"h_out aliases h0 M={M} {act}")
        prob = W.random_problem(seed, 4, 8192 + 77, 256, M, act=act, gamma_range=(1e-5, 1.0),
                                gamma_log=True, with_h0=True)
        x = dev_act(prob["x"], act)
        pr = params_dev(prob)
        h0 = dev_f32(prob["h0"])
        y1, h1 = ops.resonator_mix_fwd(x, *pr, h0=h0.clone(), return_state=True)
        st = h0.clone()
        y2 = ops.resonator_mix_fwd(x, *pr, h0=st, h_out=st)
        torch.cuda.synchronize()
        assert torch.equal(y1, y2)
        assert torch.equal(h1, st)


def test_workspace_reused_across_shapes():
    """One zero-filled forward workspace serves calls of different shapes in turn
    (different numbers of chains, dtypes and mode counts): every call leaves
    status 0 and matches the oracle recurrence."""
    from paper_2607_05583_amd import ops
    shapes = [(2, 3001, 70, 5, "bf16", 51), (4, 2048, 256, 8, "f32", 52), (1, 1024, 64, 8, "bf16", 53),
              (8, 700, 256, 8, "f32", 54), (4, 2048, 256, 8, "bf16", 55), (2, 3001, 70, 5, "bf16", 56)]
    need = max(ops.workspace_bytes(ops.RES_OP_FWD, torch.float32 if act == "f32" else torch.bfloat16, B, L, D, M)
               for B, L, D, M, act, _ in shapes)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for B, L, D, M, act, seed in shapes:
        say(f"shared workspace B={B} L={L} D={D} M={M} {act}")
        prob = W.random_problem(seed, B, L, D, M, act=act, gamma_range=(1e-4, 1.0), gamma_log=True, with_h0=True)
        x = dev_act(prob["x"], act)
        y, hout = ops.resonator_mix_fwd(x, *params_dev(prob), h0=dev_f32(prob["h0"]), ws=ws, return_state=True)
        assert ops.resonator_fwd_status(ws) == 0
        yr, hr = O.mix_recurrence(act64(prob["x"], act), *params_np(prob), h0=prob["h0"])
        assert rel_err(host(y), yr) <= tol(act, act)
        assert rel_err(host(hout), hr) <= (1e-4 if act == "f32" else 2e-2)


# Counter words of the single-pass forward's workspace (kernels.h, StreamArgs):
# a 256-byte header, then four 32-bit words per chain (next ticket, arrived
# work-groups, tile order, finished work-groups).
def _set_chain_word(ws, chain, j, value):
    ws.view(torch.int32)[(256 + 16 * chain + 4 * j) // 4] = value


def _chain_g(nchains, P):
    """Work-groups per chain, as the host sizes the grid (one per compute unit)."""
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    return 1 if nchains >= ncu else min(ncu // nchains, P)


def test_stale_counters_are_reported_and_touch_nothing(monkeypatch):
    """A chain whose arrival counter is not zero at the start (a workspace not
    zero-filled) sets bit 1 of the status word and leaves that chain's outputs
    untouched; every kernel ends normally; a zero-filled workspace then gives the
    oracle's result."""
    from paper_2607_05583_amd import ops
    monkeypatch.setattr(ops, "CHECK_FWD_STATUS", False)
    B, L, D, M = 2, 2048, 128, 8  # bf16: two blocks of 64 channels, four chains
    prob = W.random_problem(61, B, L, D, M, act="bf16", gamma_range=(1e-4, 1.0), gamma_log=True)
    x = dev_act(prob["x"], "bf16")
    ws = ops.forward_workspace(torch.bfloat16, B, L, D, M, "cuda")
    _set_chain_word(ws, 0, 1, 0x7FFFFFFF)  # chain 0 = batch row 0, channels 0 .. 63
    y = torch.full((B, L, D), 7.0, dtype=torch.bfloat16, device="cuda")
    ops.resonator_mix_fwd(x, *params_dev(prob), out=y, ws=ws)
    st = ops.resonator_fwd_status(ws)
    assert st & 2
    assert bool((y[0, :, :64] == 7.0).all())
    yr, _ = O.mix_recurrence(act64(prob["x"], "bf16"), *params_np(prob))
    assert rel_err(host(y[1]), yr[1]) <= 2e-2
    ws.zero_()
    y2 = ops.resonator_mix_fwd(x, *params_dev(prob), ws=ws)
    assert ops.resonator_fwd_status(ws) == 0
    assert rel_err(host(y2), yr) <= 2e-2


def test_forced_give_up_is_reported(monkeypatch):
    """A chain whose counters say that it takes its segments by ticket and that
    segment 0 is already taken: no work-group processes segment 0, so the
    look-back of every later segment waits for an aggregate that never comes; the
    bounded wait gives up, one work-group draws a ticket past the last segment,
    the call ends, and the status word has bit 0 (a wait gave up) and bit 1
    (stale counters)."""
    from paper_2607_05583_amd import ops
    monkeypatch.setattr(ops, "CHECK_FWD_STATUS", False)
    B, L, D, M = 1, 16384, 512, 8  # bf16: 8 chains (blocks of 64 channels) of 64 tiles
    nchains, P = D // 64, (L + 255) // 256
    G = _chain_g(nchains, P)
    if G < 2:
        pytest.skip("this device gives one work-group to each chain")
    prob = W.random_problem(62, B, L, D, M, act="bf16", gamma_range=(1e-4, 1.0), gamma_log=True)
    x = dev_act(prob["x"], "bf16")
    ws = ops.forward_workspace(torch.bfloat16, B, L, D, M, "cuda")
    _set_chain_word(ws, 0, 0, 1)  # next ticket: segment 1
    _set_chain_word(ws, 0, 2, 2)  # order: tickets
    ops.resonator_mix_fwd(x, *params_dev(prob), ws=ws)
    st = ops.resonator_fwd_status(ws)
    assert st & 1 and st & 2
    ws.zero_()
    y2 = ops.resonator_mix_fwd(x, *params_dev(prob), ws=ws)
    assert ops.resonator_fwd_status(ws) == 0
    yr, _ = O.mix_recurrence(act64(prob["x"], "bf16"), *params_np(prob))
    assert rel_err(host(y2), yr) <= 2e-2
