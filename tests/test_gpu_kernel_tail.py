"""GPU parity of the quadratic causal reference (the kernel-tail baseline of
Sec. 5.3) against the oracle's direct O(L^2) form, and of the mixing path
against that reference at a length where the oracle would be slow.

Tolerance 1e-4 (float32 sums of up to L products of float32 taps, fp32 configs'
bound)."""
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
