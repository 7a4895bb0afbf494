"""Build libresonator.so (HIP kernels + C ABI) for gfx950, in-tree.

Each .hip source is compiled with hipcc to an object in ``_build/`` and the
objects are linked into ``paper_2607_05583_amd/libresonator.so``.  Packed FP32
instructions are disabled for all device code.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libresonator.so")
SOURCES = ["fwd.hip", "bwd.hip", "decode.hip", "epilogue.hip", "params.hip", "quadref.hip", "gemm.hip", "proj.hip", "fftref.hip", "api.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: install ROCm or set HIPCC")


def flags():
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-Wno-unused-result", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include")]


def _run(cmd):
    p = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature: drop that warning.
    err = "\n".join(l for l in p.stderr.splitlines()
                    if "packed-fp32-ops" not in l and "not a recognized feature" not in l)
    return p.returncode, err


def build(verbose: bool = False) -> str:
    """Compile every source and link the library; returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    jobs = []
    for src in SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        jobs.append((src, obj, [cc, *flags(), "-c", os.path.join(CSRC, src), "-o", obj]))
    with ThreadPoolExecutor(max_workers=min(len(jobs), 4)) as ex:
        results = list(ex.map(lambda j: (j[0], _run(j[2])), jobs))
    failed = [(s, e) for s, (rc, e) in results if rc != 0]
    for s, (rc, e) in results:
        if verbose and e.strip():
            print(f"[{s}]\n{e}", file=sys.stderr)
    if failed:
        raise RuntimeError("HIP compile failed:\n" + "\n".join(f"--- {s}\n{e}" for s, e in failed))
    tmp = LIB + ".tmp"
    rc, err = _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp,
                    *[j[1] for j in jobs], "-L/opt/rocm/lib", "-lrocblas", "-lrocfft", "-Wl,-rpath,/opt/rocm/lib"])
    if rc != 0:
        raise RuntimeError("link failed:\n" + err)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
