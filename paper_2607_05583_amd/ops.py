"""PyTorch binding of the resonant mixing library.

Thin argument marshalling over the C ABI of include/resonator.h: every step of
the operator runs in the library's HIP kernels; PyTorch only provides device
memory and the current stream.  Function names follow the C entry points.

Tensors: activations [B, L, D] (float32 or bfloat16, contiguous, on the GPU);
parameters gamma, omega, amp, phase float32 [D, M]; states float32 [B, D, M, 2].
"""
from __future__ import annotations

import ctypes

import torch

from . import _lib
from ._lib import RES_BF16, RES_F32, RES_OP_BWD, RES_OP_FWD, RES_OP_STATE_INIT, check

_DT = {torch.float32: RES_F32, torch.bfloat16: RES_BF16}


def _code(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")
    return _DT[t.dtype]


def _dev(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _params(gamma, omega, amp, phase, D=None):
    ps = []
    for name, p in (("gamma", gamma), ("omega", omega), ("amp", amp), ("phase", phase)):
        _dev(p, name)
        if p.dtype != torch.float32 or p.dim() != 2:
            raise ValueError(f"{name} must be float32 [D, M]")
        ps.append(p)
    if any(p.shape != ps[0].shape for p in ps):
        raise ValueError("gamma, omega, amp and phase must have the same shape [D, M]")
    if D is not None and ps[0].shape[0] != D:
        raise ValueError(f"parameters have D={ps[0].shape[0]}, activations have D={D}")
    return ps


def workspace_bytes(op: int, act_dtype: torch.dtype, B: int, L: int, D: int, M: int) -> int:
    return int(_lib.lib().resonator_workspace_bytes(op, _DT[act_dtype], B, L, D, M))


def _workspace(op, act_dtype, B, L, D, M, device, ws=None):
    """The caller's workspace (checked for size), or a new one.  A forward
    workspace must be zero before its first forward call (the calls keep it
    reusable), so a new one is zero-filled."""
    n = workspace_bytes(op, act_dtype, B, L, D, M)
    if ws is not None:
        if ws.numel() * ws.element_size() < n:
            raise ValueError(f"workspace too small: need {n} bytes")
        return ws, n
    alloc = torch.zeros if op == RES_OP_FWD else torch.empty
    return alloc(max(n, 256), dtype=torch.uint8, device=device), n


def forward_workspace(act_dtype, B, L, D, M, device):
    """A zero-filled forward workspace for sizes (B, L, D, M), reusable across calls."""
    return torch.zeros(max(workspace_bytes(RES_OP_FWD, act_dtype, B, L, D, M), 256), dtype=torch.uint8,
                       device=device)


def resonator_fwd_status(ws) -> int:
    """The forward status word of workspace ``ws`` (bit 0: a bounded wait gave up,
    bit 1: stale counters), read and cleared; synchronises the current stream."""
    _dev(ws, "ws")
    st = ctypes.c_uint32(0)
    check(_lib.lib().resonator_fwd_status(_ptr(ws), ctypes.byref(st), _stream(ws.device)))
    return int(st.value)


# When set (the GPU tests set it), every resonator_mix_fwd reads its workspace's
# status word after the call (a synchronisation) and raises if it is not zero.
CHECK_FWD_STATUS = False


def resonator_mix_fwd(x, gamma, omega, amp, phase, h0=None, out_dtype=None, return_state=False,
                      out=None, ws=None, h_out=None):
    """y = causal resonant mixing of x (and the terminal state if return_state).

    ``h_out`` [B, D, M, 2] float32 receives the terminal state (it may be the
    ``h0`` tensor itself: the state is then advanced in place)."""
    _dev(x, "x")
    if x.dim() != 3:
        raise ValueError("x must be [B, L, D]")
    B, L, D = x.shape
    gamma, omega, amp, phase = _params(gamma, omega, amp, phase, D)
    M = gamma.shape[1]
    out_dtype = x.dtype if out_dtype is None else out_dtype
    y = out if out is not None else torch.empty((B, L, D), dtype=out_dtype, device=x.device)
    _dev(y, "out")
    if h_out is not None:
        _dev(h_out, "h_out")
        if h_out.dtype != torch.float32 or tuple(h_out.shape) != (B, D, M, 2):
            raise ValueError("h_out must be float32 [B, D, M, 2]")
    elif return_state:
        h_out = torch.empty((B, D, M, 2), dtype=torch.float32, device=x.device)
    if h0 is not None:
        _dev(h0, "h0")
        if h0.dtype != torch.float32 or tuple(h0.shape) != (B, D, M, 2):
            raise ValueError("h0 must be float32 [B, D, M, 2]")
    w, n = _workspace(RES_OP_FWD, x.dtype, B, L, D, M, x.device, ws)
    check(_lib.lib().resonator_mix_fwd(
        _ptr(x), _code(x), _ptr(y), _code(y), B, L, D, M, _ptr(gamma), _ptr(omega), _ptr(amp),
        _ptr(phase), _ptr(h0), _ptr(h_out), _ptr(w), n, _stream(x.device)))
    if CHECK_FWD_STATUS and not torch.cuda.is_current_stream_capturing():
        st = resonator_fwd_status(w)
        if st != 0:
            raise _lib.ResonatorError(_lib.RES_ERR_HIP, f"forward status word {st:#x} (bit 0: a wait gave up, "
                                                        "bit 1: stale workspace counters)")
    return (y, h_out) if return_state else y


def resonator_mix_bwd(x, dy, gamma, omega, amp, phase, h0=None, want_dh0=False, ws=None):
    """Gradients of sum(dy * y): dict with dx, dgamma, domega, damp, dphase (, dh0)."""
    _dev(x, "x")
    _dev(dy, "dy")
    if x.shape != dy.shape or x.dtype != dy.dtype or x.dim() != 3:
        raise ValueError("x and dy must have the same [B, L, D] shape and dtype")
    B, L, D = x.shape
    gamma, omega, amp, phase = _params(gamma, omega, amp, phase, D)
    M = gamma.shape[1]
    if h0 is not None:
        _dev(h0, "h0")
        if h0.dtype != torch.float32 or tuple(h0.shape) != (B, D, M, 2):
            raise ValueError("h0 must be float32 [B, D, M, 2]")
    dx = torch.empty_like(x)
    g = {k: torch.empty((D, M), dtype=torch.float32, device=x.device)
         for k in ("dgamma", "domega", "damp", "dphase")}
    dh0 = torch.empty((B, D, M, 2), dtype=torch.float32, device=x.device) if want_dh0 else None
    w, n = _workspace(RES_OP_BWD, x.dtype, B, L, D, M, x.device, ws)
    check(_lib.lib().resonator_mix_bwd(
        _ptr(x), _ptr(dy), _code(x), _ptr(dx), B, L, D, M, _ptr(gamma), _ptr(omega), _ptr(amp),
        _ptr(phase), _ptr(h0), _ptr(g["dgamma"]), _ptr(g["domega"]), _ptr(g["damp"]),
        _ptr(g["dphase"]), _ptr(dh0), _ptr(w), n, _stream(x.device)))
    out = {"dx": dx, **g}
    if want_dh0:
        out["dh0"] = dh0
    return out


def resonator_state_init(x_prompt, gamma, omega, amp, phase, out=None, ws=None):
    """Decode state after a prompt x_prompt [B, L, D] (L may be 0)."""
    _dev(x_prompt, "x_prompt")
    B, L, D = x_prompt.shape
    gamma, omega, amp, phase = _params(gamma, omega, amp, phase, D)
    M = gamma.shape[1]
    st = out if out is not None else torch.empty((B, D, M, 2), dtype=torch.float32,
                                                  device=x_prompt.device)
    if L > 0:
        w, n = _workspace(RES_OP_STATE_INIT, x_prompt.dtype, B, L, D, M, x_prompt.device, ws)
    else:
        w, n = None, 0
    check(_lib.lib().resonator_state_init(
        _ptr(x_prompt) if L > 0 else None, _code(x_prompt), B, L, D, M, _ptr(gamma), _ptr(omega),
        _ptr(amp), _ptr(phase), _ptr(st), _ptr(w), n, _stream(x_prompt.device)))
    return st


def resonator_decode_step(x_t, gamma, omega, amp, phase, state, out_dtype=None, out=None):
    """One decode step: updates state [B, D, M, 2] in place, returns y_t [B, D]."""
    _dev(x_t, "x_t")
    _dev(state, "state")
    B, D = x_t.shape
    gamma, omega, amp, phase = _params(gamma, omega, amp, phase, D)
    M = gamma.shape[1]
    if state.dtype != torch.float32 or tuple(state.shape) != (B, D, M, 2):
        raise ValueError("state must be float32 [B, D, M, 2]")
    out_dtype = x_t.dtype if out_dtype is None else out_dtype
    y = out if out is not None else torch.empty((B, D), dtype=out_dtype, device=x_t.device)
    check(_lib.lib().resonator_decode_step(
        _ptr(x_t), _code(x_t), _ptr(y), _code(y), B, D, M, _ptr(gamma), _ptr(omega), _ptr(amp),
        _ptr(phase), _ptr(state), _stream(x_t.device)))
    return y


def resonator_decode_constants(gamma, omega, amp, phase, out=None):
    """The decode constants table [D, M, 6] float32 (lambda's float32 pair hi, lo
    and c, as (Re, Im)), evaluated once for resonator_decode_step_tab."""
    gamma, omega, amp, phase = _params(gamma, omega, amp, phase)
    D, M = gamma.shape
    tab = out if out is not None else torch.empty((D, M, 6), dtype=torch.float32, device=gamma.device)
    if tab.dtype != torch.float32 or tuple(tab.shape) != (D, M, 6) or not tab.is_contiguous():
        raise ValueError("tab must be a contiguous float32 [D, M, 6] tensor")
    check(_lib.lib().resonator_decode_constants(D, M, _ptr(gamma), _ptr(omega), _ptr(amp), _ptr(phase),
                                                _ptr(tab), _stream(gamma.device)))
    return tab


def resonator_decode_step_tab(x_t, tab, state, out_dtype=None, out=None):
    """One decode step from a constants table (bitwise resonator_decode_step):
    updates state [B, D, M, 2] in place, returns y_t [B, D]."""
    _dev(x_t, "x_t")
    _dev(state, "state")
    _dev(tab, "tab")
    B, D = x_t.shape
    if tab.dtype != torch.float32 or tab.dim() != 3 or tab.shape[0] != D or tab.shape[2] != 6:
        raise ValueError("tab must be float32 [D, M, 6]")
    M = tab.shape[1]
    if state.dtype != torch.float32 or tuple(state.shape) != (B, D, M, 2):
        raise ValueError("state must be float32 [B, D, M, 2]")
    out_dtype = x_t.dtype if out_dtype is None else out_dtype
    y = out if out is not None else torch.empty((B, D), dtype=out_dtype, device=x_t.device)
    check(_lib.lib().resonator_decode_step_tab(_ptr(x_t), _code(x_t), _ptr(y), _code(y), B, D, M, _ptr(tab),
                                               _ptr(state), _stream(x_t.device)))
    return y


def resonator_decode_steps(x, gamma, omega, amp, phase, state, out_dtype=None, out=None):
    """N decode steps in one launch: x [B, N, D] drives known in advance; updates
    state [B, D, M, 2] in place and returns y [B, N, D] (bitwise N decode steps)."""
    _dev(x, "x")
    _dev(state, "state")
    B, N, D = x.shape
    gamma, omega, amp, phase = _params(gamma, omega, amp, phase, D)
    M = gamma.shape[1]
    if state.dtype != torch.float32 or tuple(state.shape) != (B, D, M, 2):
        raise ValueError("state must be float32 [B, D, M, 2]")
    out_dtype = x.dtype if out_dtype is None else out_dtype
    y = out if out is not None else torch.empty((B, N, D), dtype=out_dtype, device=x.device)
    check(_lib.lib().resonator_decode_steps(
        _ptr(x), _code(x), _ptr(y), _code(y), B, N, D, M, _ptr(gamma), _ptr(omega), _ptr(amp),
        _ptr(phase), _ptr(state), _stream(x.device)))
    return y


class DecodeGraph:
    """K decode steps (Sec. 3.3) captured once as a HIP graph and replayed: one
    token's step is a single short launch, so a replay issues the K launches of a
    block of tokens without K host round trips.

    Static buffers: ``x`` [K, B, D] holds the drives of the next K tokens (copy
    them in, or pass them to ``replay``), ``y`` [K, B, D] receives the outputs;
    ``state`` [B, D, M, 2] is updated in place by every replay.  The parameters
    and the state are captured by address: update them in place, never rebind
    them.  A replay first evaluates the decode constants from the parameters into
    a table (one launch), then runs the K steps from the table
    (resonator_decode_step_tab, bitwise resonator_decode_step).  The capture
    records these kernels only (no allocation, no memset), and nothing runs until
    the first replay."""

    def __init__(self, gamma, omega, amp, phase, state, steps: int, x_dtype=torch.bfloat16, out_dtype=None):
        _dev(state, "state")
        gamma, omega, amp, phase = _params(gamma, omega, amp, phase)
        D, M = gamma.shape
        if state.dtype != torch.float32 or state.dim() != 4 or tuple(state.shape[1:]) != (D, M, 2):
            raise ValueError("state must be float32 [B, D, M, 2]")
        if steps < 1:
            raise ValueError("steps must be >= 1")
        B = state.shape[0]
        dev = state.device
        out_dtype = x_dtype if out_dtype is None else out_dtype
        self.params = (gamma, omega, amp, phase)
        self.state = state
        self.x = torch.zeros((steps, B, D), dtype=x_dtype, device=dev)
        self.y = torch.empty((steps, B, D), dtype=out_dtype, device=dev)
        self.tab = torch.empty((D, M, 6), dtype=torch.float32, device=dev)
        _lib.lib()  # loaded before the capture
        self.graph = torch.cuda.CUDAGraph()
        cur = torch.cuda.current_stream(dev)
        cap = torch.cuda.Stream(dev)
        cap.wait_stream(cur)
        with torch.cuda.stream(cap), torch.cuda.graph(self.graph, stream=cap):
            resonator_decode_constants(*self.params, out=self.tab)
            for k in range(steps):
                resonator_decode_step_tab(self.x[k], self.tab, state, out=self.y[k])
        cur.wait_stream(cap)

    def replay(self, x=None):
        """Run the K steps on the current stream (after copying ``x`` [K, B, D] into
        the drive buffer when given); returns the output buffer ``y``."""
        if x is not None:
            self.x.copy_(x)
        self.graph.replay()
        return self.y


def resonator_quadratic_reference(x, gamma, omega, amp, phase):
    """The O(L^2) direct causal mixer (kernel-tail baseline), float32 [B, L, D]."""
    _dev(x, "x")
    if x.dtype != torch.float32 or x.dim() != 3:
        raise ValueError("x must be float32 [B, L, D]")
    B, L, D = x.shape
    gamma, omega, amp, phase = _params(gamma, omega, amp, phase, D)
    M = gamma.shape[1]
    y = torch.empty_like(x)
    n = _lib.lib().resonator_quadratic_reference_workspace_bytes(L, D)
    ws = torch.empty(max(n, 4), dtype=torch.uint8, device=x.device)
    check(_lib.lib().resonator_quadratic_reference(_ptr(x), _ptr(y), B, L, D, M, _ptr(gamma), _ptr(omega),
                                                   _ptr(amp), _ptr(phase), _ptr(ws), n, _stream(x.device)))
    return y


def resonator_fft_reference(x, gamma, omega, amp, phase):
    """The mixing by zero-padded FFT convolution (the paper's prefill form), float32 [B, L, D]."""
    _dev(x, "x")
    if x.dtype != torch.float32 or x.dim() != 3:
        raise ValueError("x must be float32 [B, L, D]")
    B, L, D = x.shape
    gamma, omega, amp, phase = _params(gamma, omega, amp, phase, D)
    M = gamma.shape[1]
    y = torch.empty_like(x)
    n = _lib.lib().resonator_fft_reference_workspace_bytes(B, L, D)
    if n == 0:
        raise _lib.ResonatorError(0, "FFT workspace query failed: "
                                  + _lib.lib().resonator_last_error().decode(errors="replace"))
    ws = torch.empty(n, dtype=torch.uint8, device=x.device)
    check(_lib.lib().resonator_fft_reference(_ptr(x), _ptr(y), B, L, D, M, _ptr(gamma), _ptr(omega),
                                             _ptr(amp), _ptr(phase), _ptr(ws), n, _stream(x.device)))
    return y


def resonator_grouped_linear(x, W, out=None):
    """y = x W for a block-diagonal W of G groups: x [..., d_in], W [G, d_in/G, d_out/G]."""
    _dev(x, "x")
    _dev(W, "W")
    if W.dim() != 3 or W.dtype != x.dtype:
        raise ValueError("W must be [G, d_in/G, d_out/G] of x's dtype")
    G, di, dq = W.shape
    d_in = x.shape[-1]
    if d_in != G * di:
        raise ValueError(f"x has {d_in} features, W expects {G * di}")
    N = x.numel() // d_in
    y = out if out is not None else torch.empty(x.shape[:-1] + (G * dq,), dtype=x.dtype, device=x.device)
    _dev(y, "out")
    check(_lib.lib().resonator_grouped_linear(_ptr(x), _ptr(W), _code(x), _ptr(y), N, d_in, G * dq, G,
                                              _stream(x.device)))
    return y


def resonator_grouped_linear2(x, W0, W1, out0=None, out1=None):
    """y0 = x W0 and y1 = x W1 for block-diagonal weights of one shape (the drive
    and the gate of Sec. 3.1), from one read of x.  Returns (y0, y1)."""
    _dev(x, "x")
    _dev(W0, "W0")
    _dev(W1, "W1")
    if W0.dim() != 3 or W0.dtype != x.dtype or W1.shape != W0.shape or W1.dtype != x.dtype:
        raise ValueError("W0 and W1 must both be [G, d_in/G, d_out/G] of x's dtype")
    G, di, dq = W0.shape
    d_in = x.shape[-1]
    if d_in != G * di:
        raise ValueError(f"x has {d_in} features, W expects {G * di}")
    N = x.numel() // d_in
    shape = x.shape[:-1] + (G * dq,)
    y0 = out0 if out0 is not None else torch.empty(shape, dtype=x.dtype, device=x.device)
    y1 = out1 if out1 is not None else torch.empty(shape, dtype=x.dtype, device=x.device)
    _dev(y0, "out0")
    _dev(y1, "out1")
    check(_lib.lib().resonator_grouped_linear2(_ptr(x), _ptr(W0), _ptr(W1), _code(x), _ptr(y0), _ptr(y1), N, d_in,
                                               G * dq, G, _stream(x.device)))
    return y0, y1


def resonator_grouped_linear_bwd(x, W, dy, dx=None, dW=None, accumulate=False):
    """Gradients of sum(dy * grouped_linear(x, W)): (dx of x's dtype, dW float32).

    With ``accumulate`` the gradients are added into the given ``dx``/``dW``; pass
    x = None to skip dW, W = None to skip dx."""
    ref = x if x is not None else dy
    _dev(dy, "dy")
    _code(dy)
    d_out = dy.shape[-1]
    N = dy.numel() // d_out
    if W is not None:
        _dev(W, "W")
        if W.dtype != dy.dtype or W.dim() != 3 or W.shape[0] * W.shape[2] != d_out:
            raise ValueError("W must be [G, d_in/G, d_out/G] of dy's dtype")
        G, di, dq = W.shape
        if dx is not None:
            _dev(dx, "dx")
            if dx.dtype != dy.dtype or dx.numel() != N * G * di:
                raise ValueError("dx must have dy's dtype and [N, d_in] elements")
        if dx is None:
            dx = torch.empty(dy.shape[:-1] + (G * di,), dtype=dy.dtype, device=dy.device)
        check(_lib.lib().resonator_grouped_linear_bwd_data(_ptr(dy), _ptr(W), _code(dy), _ptr(dx), N, G * di, d_out, G,
                                                           int(accumulate), _stream(dy.device)))
    if x is not None:
        _dev(x, "x")
        d_in = x.shape[-1]
        if x.dtype != dy.dtype or x.numel() != N * d_in:
            raise ValueError("x must have dy's dtype and the same number of rows")
        G = (W.shape[0] if W is not None else None) if dW is None else dW.shape[0]
        if G is None:
            raise ValueError("need W or dW to know the groups")
        if d_in % G or d_out % G:
            raise ValueError("d_in and d_out must be multiples of the group count")
        if dW is None:
            dW = torch.empty((G, d_in // G, d_out // G), dtype=torch.float32, device=ref.device)
        else:
            _dev(dW, "dW")
            if dW.dtype != torch.float32 or tuple(dW.shape) != (G, d_in // G, d_out // G):
                raise ValueError("dW must be float32 [G, d_in/G, d_out/G]")
        check(_lib.lib().resonator_grouped_linear_bwd_weight(_ptr(x), _ptr(dy), _code(x), _ptr(dW), N, d_in, d_out, G,
                                                             int(accumulate), _stream(dy.device)))
    return dx, dW


def grouped_dgrad_supported(n, d_in, d_out, G, dtype) -> bool:
    """Whether resonator_grouped_linear_bwd_data_sum runs the library's MFMA
    kernel for n gradients of this shape (16-byte aligned tensors assumed):
    d_out/G a multiple of 32 (bf16) or 16 (float32), d_in/G a multiple of 16 and
    at most 128, d_out at most 256 elements (512 bytes with n = 1), and the n
    weights at most 64 KB."""
    bf = dtype == torch.bfloat16
    kc, es = (32, 2) if bf else (16, 4)
    if not 1 <= n <= 3 or d_in % G or d_out % G:
        return False
    di, dq = d_in // G, d_out // G
    if dq % kc or di % 16 or di > 128:
        return False
    if d_out // kc > (16 if n == 1 else 8):
        return False
    return n * G * (dq // kc) * (di // 16) * 1024 <= 64 * 1024


def resonator_grouped_linear_bwd_data_sum(dys, Ws, dx=None, accumulate=False):
    """dx = sum_k dys[k] W_k^T per group (the data gradients of up to three
    grouped projections of one input, summed in float32 and rounded once); with
    ``accumulate`` added to the given ``dx``.  Returns dx."""
    if not 1 <= len(dys) <= 3 or len(dys) != len(Ws):
        raise ValueError("need 1 to 3 gradients, one weight each")
    dy0 = dys[0]
    _dev(dy0, "dy")
    _code(dy0)
    d_out = dy0.shape[-1]
    N = dy0.numel() // d_out
    G, di, dq = Ws[0].shape
    for k, (d_, W) in enumerate(zip(dys, Ws)):
        _dev(d_, f"dys[{k}]")
        _dev(W, f"Ws[{k}]")
        if d_.dtype != dy0.dtype or tuple(d_.shape) != tuple(dy0.shape):
            raise ValueError("every gradient must have the first one's dtype and shape")
        if W.dtype != dy0.dtype or tuple(W.shape) != (G, di, dq) or G * dq != d_out:
            raise ValueError("every W must be [G, d_in/G, d_out/G] of the gradients' dtype")
    if dx is None:
        dx = torch.empty(dy0.shape[:-1] + (G * di,), dtype=dy0.dtype, device=dy0.device)
    else:
        _dev(dx, "dx")
        if dx.dtype != dy0.dtype or dx.numel() != N * G * di:
            raise ValueError("dx must have the gradients' dtype and [N, d_in] elements")
    n = len(dys)
    arr = ctypes.c_void_p * n
    check(_lib.lib().resonator_grouped_linear_bwd_data_sum(n, arr(*[_ptr(d_) for d_ in dys]),
                                                           arr(*[_ptr(W) for W in Ws]), _code(dy0), _ptr(dx), N,
                                                           G * di, d_out, G, int(accumulate), _stream(dy0.device)))
    return dx


def grouped_wgrad_supported(n, nout, d_in, d_out, G, dtype) -> bool:
    """Whether resonator_grouped_linear_bwd_weight_sum runs the library's MFMA
    kernel for this shape (16-byte aligned x and gradients assumed): bf16, d_in
    and d_out multiples of 64 up to 256, d_in/G and d_out/G multiples of 16, at
    most 64 output blocks of 16 x 16."""
    return _lib.lib().resonator_grouped_linear_bwd_weight_sum_workspace_bytes(
        n, nout, 1, d_in, d_out, G, RES_BF16 if dtype == torch.bfloat16 else RES_F32) > 0


def resonator_grouped_linear_bwd_weight_sum(x, dys, outs, dWs, accumulate=False):
    """Weight gradients dWs[m] (float32 [G, d_in/G, d_out/G]) of grouped
    projections of x: dWs[m] (+)= sum over k with outs[k] = m of x^T dys[k] per
    group, in one pass over x (the library's MFMA kernel where it takes the shape;
    deterministic).  Returns dWs."""
    _dev(x, "x")
    _code(x)
    n = len(dys)
    if not 1 <= n <= 3 or len(outs) != n or not 1 <= len(dWs) <= 2:
        raise ValueError("need 1 to 3 gradients with one weight index each, and 1 or 2 weights")
    if any(o not in (0, 1) or o >= len(dWs) for o in outs) or 0 not in outs or (len(dWs) == 2 and 1 not in outs):
        raise ValueError("outs must name every given weight (indices 0 or 1)")
    d_in = x.shape[-1]
    N = x.numel() // d_in
    d_out = dys[0].shape[-1]
    for k, d_ in enumerate(dys):
        _dev(d_, f"dys[{k}]")
        if d_.dtype != x.dtype or d_.numel() != N * d_out or d_.shape[-1] != d_out:
            raise ValueError("every gradient must have x's dtype, x's rows and one width")
    G = dWs[0].shape[0]
    for m, dW in enumerate(dWs):
        _dev(dW, f"dWs[{m}]")
        if dW.dtype != torch.float32 or G < 1 or d_in % G or d_out % G or tuple(dW.shape) != (G, d_in // G, d_out // G):
            raise ValueError(f"dWs[{m}] must be float32 [G, d_in/G, d_out/G]")
    nout = len(dWs)
    nb = _lib.lib().resonator_grouped_linear_bwd_weight_sum_workspace_bytes(n, nout, N, d_in, d_out, G, _code(x))
    ws = torch.empty(max(nb, 256), dtype=torch.uint8, device=x.device)
    arr = ctypes.c_void_p * n
    check(_lib.lib().resonator_grouped_linear_bwd_weight_sum(
        n, _ptr(x), arr(*[_ptr(d_) for d_ in dys]), (ctypes.c_int * n)(*outs), _code(x), _ptr(dWs[0]),
        _ptr(dWs[1]) if nout == 2 else None, N, d_in, d_out, G, int(accumulate), _ptr(ws), ws.numel(),
        _stream(x.device)))
    return dWs


def resonator_grouped_linear_bwd_weight_split(x, dy, dW, accumulate=False):
    """Grouped weight gradient dW [G, d_in/G, d_out/G] (float32) of a long
    contraction, split into chunks (dense partial products, then their diagonal
    blocks summed in a fixed order); the same result as the unsplit form."""
    _dev(x, "x")
    _dev(dy, "dy")
    _dev(dW, "dW")
    _code(x)
    d_in, d_out = x.shape[-1], dy.shape[-1]
    N = x.numel() // d_in
    if dy.dtype != x.dtype:
        raise ValueError(f"dy must have x's dtype ({x.dtype}), got {dy.dtype}")
    if dy.numel() != N * d_out:
        raise ValueError("x and dy must have the same number of rows")
    if dW.dtype != torch.float32 or dW.dim() != 3:
        raise ValueError("dW must be float32 [G, d_in/G, d_out/G]")
    G = dW.shape[0]
    if G < 1 or d_in % G or d_out % G or tuple(dW.shape) != (G, d_in // G, d_out // G):
        raise ValueError(f"dW must be [G, d_in/G, d_out/G] = [{G}, {d_in}/{G}, {d_out}/{G}]")
    n = _lib.lib().resonator_grouped_linear_bwd_weight_split_workspace_bytes(N, d_in, d_out)
    ws = torch.empty(max(n, 256), dtype=torch.uint8, device=x.device)
    check(_lib.lib().resonator_grouped_linear_bwd_weight_split(_ptr(x), _ptr(dy), _code(x), _ptr(dW), N, d_in, d_out,
                                                               dW.shape[0], int(accumulate), _ptr(ws), n,
                                                               _stream(x.device)))
    return dW


def resonator_block_diag_weight(W):
    """Dense [1, d_in, d_out] block-diagonal copy of a grouped weight [G, d_in/G, d_out/G]."""
    _dev(W, "W")
    G, di, dq = W.shape
    Wd = torch.empty((1, G * di, G * dq), dtype=W.dtype, device=W.device)
    check(_lib.lib().resonator_block_diag_weight(_ptr(W), _code(W), G * di, G * dq, G, _ptr(Wd), _stream(W.device)))
    return Wd


def resonator_block_diag_extract(Wd, G, out=None, accumulate=False):
    """The G diagonal blocks of a dense float32 [.., d_in, d_out] matrix as
    [G, d_in/G, d_out/G] (added into ``out`` when ``accumulate``)."""
    _dev(Wd, "W_dense")
    if Wd.dtype != torch.float32 or Wd.dim() < 2:
        raise ValueError("W_dense must be float32 [..., d_in, d_out]")
    d_in, d_out = Wd.shape[-2], Wd.shape[-1]
    if Wd.numel() != d_in * d_out:
        raise ValueError("W_dense must hold one d_in x d_out matrix")
    W = out if out is not None else torch.empty((G, d_in // G, d_out // G), dtype=torch.float32, device=Wd.device)
    if out is not None:
        _dev(out, "out")
    check(_lib.lib().resonator_block_diag_extract(_ptr(Wd), d_in, d_out, G, _ptr(W), int(accumulate),
                                                  _stream(Wd.device)))
    return W


def resonator_block_fwd(x, Wu, Wg, Wo, gamma, omega, amp, phase, Ct, lambda_c, w, s, H, dense=None, save=False):
    """The mixer block forward (Sec. 3.1, 3.4): drive u and gate g from grouped
    projections of x, y = mixing of u, z = sigmoid(g) (C y) + s conv(u), and the
    grouped output projection of z.  x [B, L, d]; returns [B, L, d_out].

    Without ``dense`` the drive and the gate come from one grouped projection
    call (one read of x), the projections run grouped (the library's MFMA
    kernel where the shape allows), and with one output group per head the
    epilogue runs fused into the output projection (z is never written).
    ``dense`` = (Wu, Wg, Wo) as resonator_block_diag_weight copies: the
    projections then run as dense GEMMs and the epilogue on its own (the same
    result up to the order of float32 sums).

    With ``save`` returns (out, saved): saved = dict(u, g, y, z), the forward's
    intermediates, for resonator_block_bwd(..., saved=saved) to use instead of
    recomputing them (u, g and y are written by the forward anyway; the fused
    epilogue also writes z)."""
    if dense is None:
        u, g = resonator_grouped_linear2(x, Wu, Wg)
        y = resonator_mix_fwd(u, gamma, omega, amp, phase)
        K = 0 if w is None else int(w.shape[1])
        if epilogue_proj_supported(y, H, K, Wo):
            z = torch.empty_like(y) if save else None
            out = resonator_epilogue_proj_fwd(y, g, u, Ct, lambda_c, w, s, H, Wo, z=z)
        else:
            z = resonator_epilogue_fwd(y, g, u, Ct, lambda_c, w, s, H)
            out = resonator_grouped_linear(z, Wo)
        return (out, dict(u=u, g=g, y=y, z=z)) if save else out
    Pu, Pg, Po = dense
    u = resonator_grouped_linear(x, Pu)
    g = resonator_grouped_linear(x, Pg)
    y = resonator_mix_fwd(u, gamma, omega, amp, phase)
    z = resonator_epilogue_fwd(y, g, u, Ct, lambda_c, w, s, H)
    out = resonator_grouped_linear(z, Po)
    return (out, dict(u=u, g=g, y=y, z=z)) if save else out


class BlockForwardGraph:
    """The mixer block forward (``resonator_block_fwd``) for one fixed shape,
    captured once as a HIP graph and replayed: at short lengths the block's
    launches cost more host time than device time.

    ``x`` is a static input buffer (copy new inputs in, or pass them to
    ``replay``); the output and the intermediates live in the graph's memory
    pool and are overwritten by every replay.  Weights and mode parameters are
    captured by address (update them in place, never rebind them); ``lambda_c``
    and ``H`` are fixed at capture.  One eager call before the capture loads the
    library and sizes the GEMM library's workspace, so the capture records
    kernel launches only."""

    def __init__(self, x, Wu, Wg, Wo, gamma, omega, amp, phase, Ct, lambda_c, w, s, H, dense=None):
        _dev(x, "x")
        self.x = x.clone()
        self._args = (Wu, Wg, Wo, gamma, omega, amp, phase, Ct, lambda_c, w, s, H)
        self._dense = dense
        dev = x.device
        cur = torch.cuda.current_stream(dev)
        resonator_block_fwd(self.x, *self._args, dense=dense)
        torch.cuda.synchronize(dev)
        self.graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream(dev)
        cap.wait_stream(cur)
        with torch.cuda.stream(cap), torch.cuda.graph(self.graph, stream=cap):
            self.out = resonator_block_fwd(self.x, *self._args, dense=dense)
        cur.wait_stream(cap)

    def replay(self, x=None):
        """Run the block on the current stream (after copying ``x`` into the input
        buffer when given); returns the output buffer."""
        if x is not None:
            self.x.copy_(x)
        self.graph.replay()
        return self.out


def resonator_block_bwd(x, Wu, Wg, Wo, gamma, omega, amp, phase, Ct, lambda_c, w, s, H, do, dense=None, saved=None):
    """Gradients of sum(do * resonator_block_fwd(...)): the forward's intermediates
    are recomputed, then the chain rule runs backwards through the output
    projection, the epilogue, the mixing and the two input projections.  Returns
    a dict: dx, dWu, dWg, dWo (float32), dgamma, domega, damp, dphase, dCt,
    dlambda_c, dw, ds.  The intermediates come from the grouped projections and
    the data gradients from resonator_grouped_linear_bwd_data_sum (dx in one
    pass over the drive's and the gate's gradients); ``dense`` (as for
    resonator_block_fwd) runs the weight gradients with the contraction split,
    and the data gradients as dense GEMMs where the grouped kernel does not
    take the shape.  ``saved`` (from resonator_block_fwd(..., save=True) on the
    same inputs) supplies u, g, y and z instead of the recomputation."""
    _dev(x, "x")
    _dev(do, "do")
    if do.dtype != x.dtype:
        raise ValueError(f"do must have x's dtype ({x.dtype}), got {do.dtype}")
    d_out = Wo.shape[0] * Wo.shape[2]
    if tuple(do.shape) != tuple(x.shape[:-1]) + (d_out,):
        raise ValueError(f"do must be {tuple(x.shape[:-1]) + (d_out,)}, got {tuple(do.shape)}")
    Pu, Pg, Po = dense if dense is not None else (Wu, Wg, Wo)
    # the forward's intermediates from the grouped projections (one read of x
    # for the drive and the gate)
    if saved is not None:
        u, g, y, z = saved["u"], saved["g"], saved["y"], saved["z"]
        for k, t in (("u", u), ("g", g), ("y", y), ("z", z)):
            _dev(t, f"saved[{k!r}]")
            if t.dtype != x.dtype or t.shape[:-1] != x.shape[:-1]:
                raise ValueError(f"saved[{k!r}] does not come from a forward of this input")
    else:
        u, g = resonator_grouped_linear2(x, Wu, Wg)
        y = resonator_mix_fwd(u, gamma, omega, amp, phase)
        z = resonator_epilogue_fwd(y, g, u, Ct, lambda_c, w, s, H)

    def wgrad(xin, dys, Wt):
        # grouped weight gradient of the sum over dys; on the dense route with
        # the contraction split (dense partial products, then diagonal blocks)
        dW = torch.empty_like(Wt, dtype=torch.float32)
        for i, d_ in enumerate(dys):
            if dense is None:
                resonator_grouped_linear_bwd(xin, None, d_, dW=dW, accumulate=i > 0)
            else:
                resonator_grouped_linear_bwd_weight_split(xin, d_, dW, accumulate=i > 0)
        return dW

    def dgrad(dys, Ws, Ps):
        # data gradient summed over the uses of one input: the library's grouped
        # kernel where it takes the shape, else the dense GEMMs when given
        if dense is None or grouped_dgrad_supported(len(dys), Ws[0].shape[0] * Ws[0].shape[1],
                                                    Ws[0].shape[0] * Ws[0].shape[2], Ws[0].shape[0], x.dtype):
            return resonator_grouped_linear_bwd_data_sum(dys, Ws)
        dxs, _ = resonator_grouped_linear_bwd(None, Ps[0], dys[0])
        for d_, P in zip(dys[1:], Ps[1:]):
            resonator_grouped_linear_bwd(None, P, d_, dx=dxs, accumulate=True)
        return dxs

    dz = dgrad([do], [Wo], [Po])
    if grouped_wgrad_supported(1, 1, z.shape[-1], do.shape[-1], Wo.shape[0], z.dtype):
        dWo = resonator_grouped_linear_bwd_weight_sum(z, [do], [0], [torch.empty_like(Wo, dtype=torch.float32)])[0]
    else:
        dWo = wgrad(z, [do], Wo)
    dy, dg, dv, dCt, dlam, dw, ds = resonator_epilogue_bwd(y, g, u, dz, Ct, lambda_c, w, s, H)
    mb = resonator_mix_bwd(u, dy, gamma, omega, amp, phase)
    # du = mb["dx"] + dv enters both the data and the weight gradient of W_u;
    # dx sums the data gradients through W_u (twice) and W_g in one pass, and
    # dW_u, dW_g come from one pass over x
    dus = [mb["dx"]] + ([dv] if dv is not None else [])
    dx = dgrad(dus + [dg], [Wu] * len(dus) + [Wg], [Pu] * len(dus) + [Pg])
    if Wu.shape == Wg.shape and grouped_wgrad_supported(len(dus) + 1, 2, x.shape[-1], Wu.shape[0] * Wu.shape[2],
                                                        Wu.shape[0], x.dtype):
        dWu, dWg = resonator_grouped_linear_bwd_weight_sum(
            x, dus + [dg], [0] * len(dus) + [1],
            [torch.empty_like(Wu, dtype=torch.float32), torch.empty_like(Wg, dtype=torch.float32)])
    else:
        dWu = wgrad(x, dus, Wu)
        dWg = wgrad(x, [dg], Wg)
    return dict(dx=dx, dWu=dWu, dWg=dWg, dWo=dWo, dgamma=mb["dgamma"], domega=mb["domega"], damp=mb["damp"],
                dphase=mb["dphase"], dCt=dCt, dlambda_c=dlam, dw=dw, ds=ds)


ALPHA_MIN = 1e-4  # the paper's floor on the damping


def _f32_pair(a, b, name_a, name_b):
    _dev(a, name_a)
    _dev(b, name_b)
    if a.dtype != torch.float32 or b.dtype != torch.float32 or a.shape != b.shape:
        raise ValueError(f"{name_a} and {name_b} must be float32 of one shape")


def resonator_params_map(theta_gamma, theta_omega, alpha_min=ALPHA_MIN):
    """(gamma, omega) = (alpha_min + softplus(theta_gamma), pi sigmoid(theta_omega)), Sec. 3.1."""
    _f32_pair(theta_gamma, theta_omega, "theta_gamma", "theta_omega")
    gamma, omega = torch.empty_like(theta_gamma), torch.empty_like(theta_omega)
    check(_lib.lib().resonator_params_map(_ptr(theta_gamma), _ptr(theta_omega), theta_gamma.numel(),
                                          float(alpha_min), _ptr(gamma), _ptr(omega), _stream(gamma.device)))
    return gamma, omega


def resonator_params_map_bwd(theta_gamma, theta_omega, dgamma, domega):
    """Chain rule of resonator_params_map: returns (dtheta_gamma, dtheta_omega)."""
    _f32_pair(theta_gamma, theta_omega, "theta_gamma", "theta_omega")
    _f32_pair(dgamma, domega, "dgamma", "domega")
    if dgamma.shape != theta_gamma.shape:
        raise ValueError("gradients must match the parameters in shape")
    dtg, dtw = torch.empty_like(theta_gamma), torch.empty_like(theta_omega)
    check(_lib.lib().resonator_params_map_bwd(_ptr(theta_gamma), _ptr(theta_omega), _ptr(dgamma), _ptr(domega),
                                              theta_gamma.numel(), _ptr(dtg), _ptr(dtw), _stream(dtg.device)))
    return dtg, dtw


def resonator_params_init(D, M, hl_min=2.0, hl_max=2048.0, per_min=4.0, per_max=2048.0, alpha_min=ALPHA_MIN,
                          device="cuda"):
    """Unconstrained (theta_gamma, theta_omega) [D, M] with log-spaced half-lives and periods."""
    tg = torch.empty((D, M), dtype=torch.float32, device=device)
    tw = torch.empty_like(tg)
    check(_lib.lib().resonator_params_init(D, M, float(hl_min), float(hl_max), float(per_min), float(per_max),
                                           float(alpha_min), _ptr(tg), _ptr(tw), _stream(tg.device)))
    return tg, tw


class ResonatorParamMapFunction(torch.autograd.Function):
    """Autograd wrapper of the parameter map (forward and chain rule on the GPU)."""

    @staticmethod
    def forward(ctx, theta_gamma, theta_omega, alpha_min=ALPHA_MIN):
        ctx.save_for_backward(theta_gamma, theta_omega)
        return resonator_params_map(theta_gamma.contiguous(), theta_omega.contiguous(), alpha_min)

    @staticmethod
    def backward(ctx, dgamma, domega):
        tg, tw = ctx.saved_tensors
        dtg, dtw = resonator_params_map_bwd(tg.contiguous(), tw.contiguous(), dgamma.contiguous(),
                                            domega.contiguous())
        return dtg, dtw, None


class ResonatorMixFunction(torch.autograd.Function):
    """Autograd wrapper: forward = resonator_mix_fwd, backward = resonator_mix_bwd."""

    @staticmethod
    def forward(ctx, x, gamma, omega, amp, phase):
        ctx.save_for_backward(x, gamma, omega, amp, phase)
        return resonator_mix_fwd(x.contiguous(), gamma.contiguous(), omega.contiguous(),
                                 amp.contiguous(), phase.contiguous())

    @staticmethod
    def backward(ctx, dy):
        x, gamma, omega, amp, phase = ctx.saved_tensors
        g = resonator_mix_bwd(x.contiguous(), dy.contiguous().to(x.dtype), gamma, omega, amp, phase)
        return g["dx"], g["dgamma"], g["domega"], g["damp"], g["dphase"]


def resonator_mix(x, gamma, omega, amp, phase):
    """Differentiable mixing (x and the four parameter tensors receive gradients)."""
    return ResonatorMixFunction.apply(x, gamma, omega, amp, phase)


# ---------------------------------------------------------------------------
# Mixer epilogue (Sec. 3.4: head coupling, gate, local path)
# ---------------------------------------------------------------------------
def _epi_params(Ct, w, s, H, D, K):
    _dev(Ct, "Ct")
    if Ct.dtype != torch.float32 or tuple(Ct.shape) != (H, H):
        raise ValueError("Ct must be float32 [H, H]")
    if K > 0:
        for name, p, shape in (("w", w, (D, K)), ("s", s, (D,))):
            _dev(p, name)
            if p.dtype != torch.float32 or tuple(p.shape) != shape:
                raise ValueError(f"{name} must be float32 {list(shape)}")


def resonator_epilogue_fwd(y, gate, v, Ct, lambda_c, w, s, H, out=None):
    """z = sigmoid(gate) * (C (x) I_dh) y + s * causal_depthwise_conv(v, w), C = I + lc/sqrt(H) tanh(Ct).

    y, gate, v: [B, L, D] (same dtype), D = H * dh; w: [D, K] float32 (K = w.shape[1];
    w = None or K = 0 disables the local path, and v, s may then be None).
    """
    _dev(y, "y"); _dev(gate, "gate")
    B, L, D = y.shape
    if gate.shape != y.shape or gate.dtype != y.dtype:
        raise ValueError("gate must match y in shape and dtype")
    if D % H:
        raise ValueError(f"D={D} is not a multiple of H={H}")
    K = 0 if w is None else int(w.shape[1])
    if K > 0:
        _dev(v, "v")
        if v.shape != y.shape or v.dtype != y.dtype:
            raise ValueError("v must match y in shape and dtype")
    _epi_params(Ct, w, s, H, D, K)
    z = torch.empty_like(y) if out is None else _dev(out, "out")
    check(_lib.lib().resonator_epilogue_fwd(
        _ptr(y), _ptr(gate), _ptr(v) if K else None, _code(y), _ptr(z), B, L, H, D // H, K, _ptr(Ct),
        float(lambda_c), _ptr(w) if K else None, _ptr(s) if K else None, _stream(y.device)))
    return z


def epilogue_proj_supported(y, H, K, Wo) -> bool:
    """Whether resonator_epilogue_proj_fwd takes this shape (one output group
    per head, a head of 32 bf16 or 16 float32 channels, H <= 8, K <= 4, d_out/H
    = 16 or 32; the tensors must also be 16-byte aligned)."""
    D = y.shape[-1]
    if Wo.dim() != 3 or Wo.shape[0] != H or D % H:
        return False
    dh, dq = D // H, Wo.shape[2]
    return (H <= 8 and K <= 4 and dh == (32 if y.dtype == torch.bfloat16 else 16) and Wo.shape[1] == dh
            and dq in (16, 32))


def resonator_epilogue_proj_fwd(y, gate, v, Ct, lambda_c, w, s, H, Wo, out=None, z=None):
    """The epilogue fused with the grouped output projection (one group per head):
    GL(resonator_epilogue_fwd(y, gate, v, ...), Wo) without writing z, unless a
    tensor ``z`` of y's shape is given to receive it.  Wo is [H, dh, d_out/H] of
    y's dtype; returns [B, L, d_out].  Bitwise the two separate calls; shapes it
    does not take raise (epilogue_proj_supported)."""
    _dev(y, "y"); _dev(gate, "gate"); _dev(Wo, "Wo")
    B, L, D = y.shape
    if gate.shape != y.shape or gate.dtype != y.dtype or Wo.dtype != y.dtype:
        raise ValueError("gate and Wo must have y's dtype, gate y's shape")
    if D % H:
        raise ValueError(f"D={D} is not a multiple of H={H}")
    K = 0 if w is None else int(w.shape[1])
    if K > 0:
        _dev(v, "v")
        if v.shape != y.shape or v.dtype != y.dtype:
            raise ValueError("v must match y in shape and dtype")
    _epi_params(Ct, w, s, H, D, K)
    if Wo.dim() != 3 or Wo.shape[0] != H or Wo.shape[1] != D // H:
        raise ValueError(f"Wo must be [H, dh, d_out/H] = [{H}, {D // H}, *]")
    d_out = H * Wo.shape[2]
    o = torch.empty((B, L, d_out), dtype=y.dtype, device=y.device) if out is None else _dev(out, "out")
    if z is not None:
        _dev(z, "z")
        if z.shape != y.shape or z.dtype != y.dtype:
            raise ValueError("z must match y in shape and dtype")
    check(_lib.lib().resonator_epilogue_proj_fwd(
        _ptr(y), _ptr(gate), _ptr(v) if K else None, _code(y), _ptr(Wo), _ptr(o), _ptr(z) if z is not None else None,
        B, L, H, D // H, K, d_out,
        _ptr(Ct), float(lambda_c), _ptr(w) if K else None, _ptr(s) if K else None, _stream(y.device)))
    return o


def resonator_epilogue_bwd(y, gate, v, dz, Ct, lambda_c, w, s, H, ws=None):
    """Gradients of sum(dz * z) for z = resonator_epilogue_fwd(...).

    Returns (dy, dgate, dv, dCt, dlambda_c, dw, ds); dv, dw, ds are None when K = 0.
    """
    _dev(y, "y"); _dev(gate, "gate"); _dev(dz, "dz")
    B, L, D = y.shape
    K = 0 if w is None else int(w.shape[1])
    for name, t in (("gate", gate), ("dz", dz)) + ((("v", v),) if K else ()):
        _dev(t, name)
        if t.shape != y.shape or t.dtype != y.dtype:
            raise ValueError(f"{name} must match y in shape and dtype")
    _epi_params(Ct, w, s, H, D, K)
    dy, dgate = torch.empty_like(y), torch.empty_like(y)
    dv = torch.empty_like(y) if K else None
    f32 = dict(dtype=torch.float32, device=y.device)
    dCt, dlam = torch.empty((H, H), **f32), torch.empty((1,), **f32)
    dw = torch.empty((D, K), **f32) if K else None
    ds = torch.empty((D,), **f32) if K else None
    n = _lib.lib().resonator_epilogue_workspace_bytes(B, L, H, D // H, K)
    if ws is None or ws.numel() < n:
        ws = torch.empty(n, dtype=torch.uint8, device=y.device)
    check(_lib.lib().resonator_epilogue_bwd(
        _ptr(y), _ptr(gate), _ptr(v) if K else None, _ptr(dz), _code(y), _ptr(dy), _ptr(dgate), _ptr(dv), B, L,
        H, D // H, K, _ptr(Ct), float(lambda_c), _ptr(w) if K else None, _ptr(s) if K else None, _ptr(dCt),
        _ptr(dlam), _ptr(dw), _ptr(ds), _ptr(ws), ws.numel(), _stream(y.device)))
    return dy, dgate, dv, dCt, dlam, dw, ds
