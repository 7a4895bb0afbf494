"""GPU parity of the two baselines of the mixing: the quadratic causal
reference (the kernel-tail baseline of Sec. 5.3) against the oracle's direct
O(L^2) form, and the FFT convolution (the paper's prefill form, Sec. 3.2)
against the oracle's FFT form and its direct form; and of the mixing path
against both at a length where the oracle would be slow.

Tolerance 1e-4: float32 sums of up to L products of float32 taps for the
quadratic form; for the FFT form the float32 transform error, about
3 log2(n) eps relative in the 2-norm (under 3e-6 at n = 2^14), an order of
magnitude more elementwise against the floor of the reference's RMS."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import dev_f32, host, params_dev, params_np, rel_err, say

pytestmark = pytest.mark.gpu

ops = None


def setup_module(module):
    global ops
    from paper_2607_05583_amd import ops as _ops
    ops = _ops
    assert torch.cuda.is_available(), "GPU tests need a HIP device"


@pytest.mark.parametrize("B,L,D,M,seed", [(1, 1, 1, 1, 71), (2, 130, 70, 3, 72), (1, 1000, 64, 8, 73),
                                          (3, 257, 129, 16, 74)])
def test_quadratic_reference_matches_the_direct_oracle(B, L, D, M, seed):
    say(f"quadratic reference B={B} L={L} D={D} M={M}")
    prob = W.random_problem(seed, B, L, D, M, act="f32", gamma_range=(1e-3, 0.5), gamma_log=True)
    y = ops.resonator_quadratic_reference(dev_f32(prob["x"]), *params_dev(prob))
    torch.cuda.synchronize()
    yr = O.mix_direct(prob["x"], *params_np(prob))
    err = rel_err(host(y), yr)
    say(f"  err {err:.2e}")
    assert err <= 1e-4


def test_mixing_matches_the_quadratic_reference_at_8k():
    prob = W.random_problem(75, 1, 8192, 256, 8, act="f32", gamma_range=(1e-4, 1.0), gamma_log=True)
    x = dev_f32(prob["x"])
    pr = params_dev(prob)
    yq = ops.resonator_quadratic_reference(x, *pr)
    ym = ops.resonator_mix_fwd(x, *pr)
    torch.cuda.synchronize()
    err = rel_err(host(ym), host(yq))
    say(f"  mixing vs quadratic reference at 8K: {err:.2e}")
    assert err <= 1e-4


@pytest.mark.parametrize("B,L,D,M,seed", [(1, 1, 1, 1, 81), (2, 130, 70, 3, 82), (1, 1000, 64, 8, 83),
                                          (3, 257, 129, 16, 84), (1, 4096, 33, 5, 85)])
def test_fft_reference_matches_the_fft_and_direct_oracles(B, L, D, M, seed):
    say(f"FFT reference B={B} L={L} D={D} M={M}")
    prob = W.random_problem(seed, B, L, D, M, act="f32", gamma_range=(1e-3, 0.5), gamma_log=True)
    y = host(ops.resonator_fft_reference(dev_f32(prob["x"]), *params_dev(prob)))
    torch.cuda.synchronize()
    pr = params_np(prob)
    err_fft = rel_err(y, O.mix_fft(prob["x"], *pr))
    err_dir = rel_err(y, O.mix_direct(prob["x"], *pr)) if L * L * D <= 1e9 else err_fft
    say(f"  err vs FFT oracle {err_fft:.2e}, vs direct oracle {err_dir:.2e}")
    assert err_fft <= 1e-4 and err_dir <= 1e-4


def test_fft_reference_repeated_calls_and_two_plan_shapes():
    """Cached plans: two shapes in turn, each twice, give the same results."""
    outs = []
    for seed, (B, L, D) in ((86, (2, 300, 16)), (87, (1, 700, 40)), (86, (2, 300, 16)), (87, (1, 700, 40))):
        prob = W.random_problem(seed, B, L, D, 4, act="f32", gamma_range=(1e-3, 0.5), gamma_log=True)
        outs.append(host(ops.resonator_fft_reference(dev_f32(prob["x"]), *params_dev(prob))))
    np.testing.assert_array_equal(outs[0], outs[2])
    np.testing.assert_array_equal(outs[1], outs[3])


def test_mixing_and_fft_reference_match_the_oracle_at_32k():
    """The kernel-tail shape at 32K (B1 D256 M8 float32): the mixing and the FFT
    convolution, each against the oracle recurrence (and the mixing against
    direct-sum spot checks), and against each other."""
    prob = W.random_problem(88, 1, 32768, 256, 8, act="f32", gamma_range=(1e-4, 1.0), gamma_log=True)
    x = dev_f32(prob["x"])
    pr = params_dev(prob)
    yf = host(ops.resonator_fft_reference(x, *pr))
    ym = host(ops.resonator_mix_fwd(x, *pr))
    torch.cuda.synchronize()
    yr = O.mix_recurrence(prob["x"], *params_np(prob))[0]
    em, ef, emf = rel_err(ym, yr), rel_err(yf, yr), rel_err(ym, yf)
    say(f"  at 32K: mixing vs oracle {em:.2e}, FFT vs oracle {ef:.2e}, mixing vs FFT {emf:.2e}")
    assert em <= 1e-4 and ef <= 1e-4 and emf <= 1e-4
    rng = np.random.default_rng(89)
    pos = np.stack([np.zeros(64, np.int64), np.concatenate([rng.integers(0, 32768, 60), [0, 255, 256, 32767]]),
                    rng.integers(0, 256, 64)], 1)
    yd = O.mix_direct_at(prob["x"], *params_np(prob), pos)
    den = np.maximum(np.abs(yd), np.sqrt(np.mean(yr ** 2)))
    assert float((np.abs(ym[pos[:, 0], pos[:, 1], pos[:, 2]] - yd) / den).max()) <= 1e-4
