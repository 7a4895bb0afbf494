"""The allocation-free forward (resonator_mix_fwd_noalloc) through the C ABI.

It must give what resonator_mix_fwd gives on the same inputs (the same kernels
on a static scratch instead of a caller workspace) within the forward's
tolerance (the look-back folds states along a path chosen at run time, so two
calls agree to rounding, not bitwise), and match the oracle; two calls in a row,
the second on a smaller problem, check that the scratch left by one call does
not leak into the next.  Sizes beyond the scratch are rejected before anything
is launched.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import act64, dev_act, dev_f32, host, params_dev, params_np, rel_err, say, tol

pytestmark = pytest.mark.gpu


def _lib():
    from paper_2607_05583_amd import _lib as L
    return L


def _noalloc(x, y, pr, h0=None, h_out=None):
    L = _lib()
    B, Ln, D = x.shape
    M = pr[0].shape[1]
    code = {torch.float32: L.RES_F32, torch.bfloat16: L.RES_BF16}
    p = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return L.lib().resonator_mix_fwd_noalloc(p(x), code[x.dtype], p(y), code[y.dtype], B, Ln, D, M,
                                              *[p(t) for t in pr], p(h0), p(h_out), st)


@pytest.mark.parametrize("act,out", [("bf16", "bf16"), ("f32", "f32"), ("bf16", "f32")])
def test_noalloc_matches_the_workspace_forward_twice(act, out):
    from paper_2607_05583_amd import ops
    L = _lib()
    assert L.lib().resonator_mix_fwd_noalloc_max_bytes() == 32 << 20
    od = torch.float32 if out == "f32" else torch.bfloat16
    for B, Ln, D, M, seed in ((4, 32768, 256, 8, 201), (2, 3001, 70, 5, 202)):
        say(f"noalloc B={B} L={Ln} D={D} M={M} {act}->{out}")
        prob = W.random_problem(seed, B, Ln, D, M, act=act, gamma_range=(1e-5, 1.0), gamma_log=True,
                                with_h0=True)
        x = dev_act(prob["x"], act)
        pr = params_dev(prob)
        h0 = dev_f32(prob["h0"])
        y_ref, h_ref = ops.resonator_mix_fwd(x, *pr, h0=h0, out_dtype=od, return_state=True)
        y = torch.full((B, Ln, D), float("nan"), dtype=od, device="cuda")
        h = torch.full((B, D, M, 2), float("nan"), dtype=torch.float32, device="cuda")
        rc = _noalloc(x, y, pr, h0=h0, h_out=h)
        assert rc == L.RES_OK, L.lib().resonator_last_error()
        torch.cuda.synchronize()
        assert rel_err(host(y), host(y_ref)) <= tol(act, out)
        assert rel_err(host(h), host(h_ref)) <= (1e-4 if act == "f32" else 2e-2)
        if Ln <= 4096:
            yr, hr = O.mix_recurrence(act64(prob["x"], act), *params_np(prob), h0=prob["h0"])
            assert rel_err(host(y), yr) <= tol(act, out)
            assert rel_err(host(h), hr) <= (1e-4 if act == "f32" else 2e-2)


def test_noalloc_rejects_sizes_beyond_the_scratch():
    L = _lib()
    B, Ln, D, M = 64, 1 << 16, 512, 8
    need = L.lib().resonator_workspace_bytes(L.RES_OP_FWD, L.RES_BF16, B, Ln, D, M)
    assert need > L.lib().resonator_mix_fwd_noalloc_max_bytes()
    fake = ctypes.c_void_p(0x7F0000000000)
    fake2 = ctypes.c_void_p(0x7F8000000000)
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = L.lib().resonator_mix_fwd_noalloc(fake, L.RES_BF16, fake2, L.RES_BF16, B, Ln, D, M,
                                           fake, fake, fake, fake, None, None, st)
    assert rc == L.RES_ERR_WORKSPACE
    assert b"static scratch" in L.lib().resonator_last_error()
