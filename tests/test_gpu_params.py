"""GPU parity of the constrained parameterization, its initialization and the
physics diagnostics (Sec. 3.1 last paragraph, Sec. 3.5) against the CPU oracle,
through the C ABI.

Tolerances: the maps run in float32 (expf / log1pf, a few ulp) on float32
inputs, so 2e-6 relative; the initialization runs in float64 and rounds once,
so 1e-6; the impulse response is the float32 forward path, 1e-4 as for the
fp32 mixing configs.  The causality check must be exactly zero.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import host, params_dev, params_np, rel_err, say

pytestmark = pytest.mark.gpu

ops = None
diag = None


def setup_module(module):
    global ops, diag
    from paper_2607_05583_amd import ops as _ops, diagnostics as _diag
    ops, diag = _ops, _diag
    assert torch.cuda.is_available(), "GPU tests need a HIP device"


def _thetas(seed, n):
    r = np.random.default_rng(seed)
    t = r.normal(scale=6.0, size=(2, n)).astype(np.float32)
    edge = np.array([0.0, -60.0, 60.0, -30.0, 30.0, 1e-3, -1e-3], dtype=np.float32)[:n]
    t[:, :len(edge)] = edge
    return t[0], t[1]


@pytest.mark.parametrize("n,alpha_min", [(1, 1e-4), (2048, 1e-4), (1000, 0.0), (4099, 0.3)])
def test_params_map_parity(n, alpha_min):
    say(f"params map n={n} alpha_min={alpha_min}")
    tg, tw = _thetas(n, n)
    g, w = ops.resonator_params_map(torch.from_numpy(tg).cuda(), torch.from_numpy(tw).cuda(), alpha_min)
    torch.cuda.synchronize()
    gr, wr = O.params_map(tg, tw, np.float32(alpha_min))
    assert rel_err(host(g), gr) <= 2e-6
    assert np.all(np.abs(host(w) - wr) <= 2e-6 * np.abs(wr) + 1e-30)
    assert np.all(host(g) >= np.float32(alpha_min)) and np.all(host(w) > 0) and np.all(host(w) < math.pi + 1e-6)


@pytest.mark.parametrize("n", [1, 777, 4096])
def test_params_map_bwd_parity(n):
    say(f"params map bwd n={n}")
    tg, tw = _thetas(100 + n, n)
    r = np.random.default_rng(n)
    dg, dw = r.normal(size=(2, n)).astype(np.float32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    dtg, dtw = ops.resonator_params_map_bwd(dev(tg), dev(tw), dev(dg), dev(dw))
    torch.cuda.synchronize()
    rg, rw = O.params_map_bwd(tg, tw, dg, dw)
    assert np.all(np.abs(host(dtg) - rg) <= 2e-6 * np.abs(rg) + 1e-30)
    assert np.all(np.abs(host(dtw) - rw) <= 2e-6 * np.abs(rw) + 1e-30)


def test_autograd_through_the_map():
    tg, tw = _thetas(7, 300)
    a = torch.from_numpy(tg).cuda().requires_grad_(True)
    b = torch.from_numpy(tw).cuda().requires_grad_(True)
    g, w = ops.ResonatorParamMapFunction.apply(a, b)
    wg = torch.linspace(-1, 1, 300, device="cuda")
    (g * wg + w * wg.flip(0)).sum().backward()
    rg, rw = O.params_map_bwd(tg, tw, host(wg), host(wg.flip(0)))
    assert np.all(np.abs(host(a.grad) - rg) <= 2e-6 * np.abs(rg) + 1e-30)
    assert np.all(np.abs(host(b.grad) - rw) <= 2e-6 * np.abs(rw) + 1e-30)


@pytest.mark.parametrize("D,M,hl,per", [(256, 8, (2.0, 2048.0), (4.0, 2048.0)), (64, 1, (2.0, 2048.0), (4.0, 2048.0)),
                                        (5, 3, (1.5, 100.0), (2.0, 50.0)), (3, 16, (10.0, 10.0), (8.0, 8.0))])
def test_params_init_parity(D, M, hl, per):
    say(f"params init D={D} M={M} hl={hl} per={per}")
    tg, tw = ops.resonator_params_init(D, M, hl[0], hl[1], per[0], per[1])
    torch.cuda.synchronize()
    rg, rw = O.params_init(D, M, hl[0], hl[1], per[0], per[1])
    assert rel_err(host(tg), rg) <= 1e-6 and rel_err(host(tw), rw) <= 1e-6
    g, w = ops.resonator_params_map(tg, tw)
    hls = host(diag.half_lives(g))
    assert abs(hls.min() / hl[0] - 1) <= 1e-4 and abs(hls.max() / hl[1] - 1) <= 1e-4


def test_params_init_rejects_half_lives_below_the_floor():
    tg = torch.empty((2, 2), device="cuda")
    with pytest.raises(Exception):
        ops.resonator_params_init(2, 2, 2.0, 1e5, 4.0, 64.0, alpha_min=1e-4, device="cuda")
    with pytest.raises(Exception):
        ops.resonator_params_init(2, 2, 2.0, 64.0, 1.0, 64.0)
    del tg


@pytest.mark.parametrize("D,M,T", [(64, 4, 1024), (7, 3, 300)])
def test_impulse_response_and_spectrum(D, M, T):
    say(f"impulse response D={D} M={M} T={T}")
    prob = W.random_problem(20 + D, 1, 8, D, M, act="f32", gamma_range=(1e-3, 0.5), gamma_log=True)
    pr = params_dev(prob)
    K = diag.impulse_response(*pr, T)
    torch.cuda.synchronize()
    Kr = O.kernel_taps(*params_np(prob), T)  # [D, T]
    Kr = Kr.T if Kr.shape == (D, T) else Kr
    assert rel_err(host(K), Kr) <= 1e-4
    # the library's closed form against the oracle's DFT of its own taps, and
    # against the FFT of the impulse response the mixing kernel produced
    S = diag.spectrum(*pr, T)
    SK = torch.fft.rfft(K, dim=0).abs()
    torch.cuda.synchronize()
    Sr = O.spectrum(*params_np(prob), T)
    assert rel_err(host(S), Sr) <= 1e-5
    assert rel_err(host(SK), Sr) <= 1e-4


def test_half_lives_and_energy_decay():
    prob = W.random_problem(31, 1, 8, 16, 4, act="f32", gamma_range=(1e-4, 1.0), gamma_log=True)
    g = torch.from_numpy(prob["gamma"]).cuda()
    assert rel_err(host(diag.half_lives(g)), O.half_lives(prob["gamma"])) <= 1e-6
    e = host(diag.energy_decay(g, 64))
    er = O.energy_decay(prob["gamma"], np.arange(64))
    assert np.all(np.abs(e - er) <= 1e-6 * np.abs(er) + 1e-37)
    with pytest.raises(Exception):
        diag.half_lives(g.double())


@pytest.mark.parametrize("act,split", [("f32", 1), ("f32", 777), ("bf16", 256), ("bf16", 4000)])
def test_causality_check_is_exact(act, split):
    say(f"causality {act} split={split}")
    prob = W.random_problem(41, 2, 4096 + 37, 64, 8, act=act, gamma_range=(1e-4, 1.0), gamma_log=True)
    from gpu_util import dev_act
    x = dev_act(prob["x"], act)
    err = diag.causality_check(x, *params_dev(prob), split)
    say(f"  max prefix change {err}")
    assert err == 0.0
