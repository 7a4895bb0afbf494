"""Causal resonant field mixing (ResonatorLM, arXiv 2607.05583) for AMD MI355X (gfx950).

The operator lives in the HIP library ``libresonator.so`` (C ABI in
``include/resonator.h``); ``paper_2607_05583_amd.ops`` is its PyTorch binding.
Importing the package does not load the library; the first call does, and
raises if it has not been built.
"""
