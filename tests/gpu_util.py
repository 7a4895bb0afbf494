"""Shared helpers of the GPU tests: device transfer of seeded inputs and the error metric."""
import sys

import numpy as np
import torch

import workloads as W

P4 = ("gamma", "omega", "amp", "phase")


def say(msg):
    """Print and flush what names the case before each GPU step."""
    print(msg, flush=True)
    sys.stdout.flush()


def dev_act(a, act: str, device="cuda"):
    """numpy activation (float32 or bf16 bits) -> torch tensor on the GPU."""
    if act == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device)


def dev_f32(a, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def params_dev(prob, device="cuda"):
    return [dev_f32(prob[k], device) for k in P4]


def params_np(prob):
    return [prob[k] for k in P4]


def act64(a, act: str) -> np.ndarray:
    return W.act_to_f32(a, act).astype(np.float64)


def rel_err(got, ref) -> float:
    """max_i |got_i - ref_i| / max(|ref_i|, rms(ref)): elementwise relative error
    with a floor at the RMS of the reference (near-zero outputs)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(ref ** 2)))
    if rms == 0.0:
        return float(np.abs(got).max())
    den = np.maximum(np.abs(ref), rms)
    return float((np.abs(got - ref) / den).max())


def tol(act: str, out: str = None) -> float:
    """Parity bounds: 1e-4 for float32 activations, 2e-2 when bf16 is involved."""
    return 1e-4 if act == "f32" and (out in (None, "f32")) else 2e-2
