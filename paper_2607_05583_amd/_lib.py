"""ctypes loader of libresonator.so (the HIP kernels behind include/resonator.h).

The library must have been built in-tree (``__graft_entry__.build()`` or
``python -m paper_2607_05583_amd._build``).  There is no fallback: if the library
is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libresonator.so")

RES_F32, RES_BF16 = 0, 1
RES_OK, RES_ERR_INVALID_ARG, RES_ERR_UNSUPPORTED, RES_ERR_MISALIGNED, RES_ERR_WORKSPACE, RES_ERR_HIP = range(6)
RES_OP_FWD, RES_OP_BWD, RES_OP_STATE_INIT = 0, 1, 2
RES_M_MAX = 16

SYMBOLS = ("resonator_version", "resonator_workspace_bytes", "resonator_mix_fwd",
           "resonator_mix_bwd", "resonator_state_init", "resonator_decode_step",
           "resonator_set_kernel_timer", "resonator_last_error", "resonator_epilogue_fwd",
           "resonator_epilogue_proj_fwd", "resonator_epilogue_bwd", "resonator_epilogue_workspace_bytes", "resonator_decode_steps",
           "resonator_decode_constants", "resonator_decode_step_tab",
           "resonator_params_map", "resonator_params_map_bwd", "resonator_params_init", "resonator_diagnostics",
           "resonator_quadratic_reference", "resonator_quadratic_reference_workspace_bytes",
           "resonator_fft_reference", "resonator_fft_reference_workspace_bytes",
           "resonator_grouped_linear", "resonator_grouped_linear2", "resonator_block_diag_weight", "resonator_block_diag_extract",
           "resonator_grouped_linear_bwd_data", "resonator_grouped_linear_bwd_data_sum",
           "resonator_grouped_linear_bwd_weight", "resonator_grouped_linear_bwd_weight_sum",
           "resonator_grouped_linear_bwd_weight_sum_workspace_bytes",
           "resonator_grouped_linear_bwd_weight_split", "resonator_grouped_linear_bwd_weight_split_workspace_bytes",
           "resonator_mix_fwd_noalloc", "resonator_mix_fwd_noalloc_max_bytes", "resonator_fwd_status",
           "resonator_fwd_status_noalloc")

_lib = None


class ResonatorError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"resonator error {code}: {msg}")
        self.code = code


def _declare(lib):
    vp, i64, i32, sz, fp = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p
    lib.resonator_version.restype = i32
    lib.resonator_version.argtypes = []
    lib.resonator_last_error.restype = ctypes.c_char_p
    lib.resonator_last_error.argtypes = []
    lib.resonator_workspace_bytes.restype = sz
    lib.resonator_workspace_bytes.argtypes = [i32, i32, i64, i64, i64, i64]
    lib.resonator_mix_fwd.restype = i32
    lib.resonator_mix_fwd.argtypes = [vp, i32, vp, i32, i64, i64, i64, i64, fp, fp, fp, fp, fp, fp,
                                      vp, sz, vp]
    lib.resonator_mix_bwd.restype = i32
    lib.resonator_mix_bwd.argtypes = [vp, vp, i32, vp, i64, i64, i64, i64, fp, fp, fp, fp, fp,
                                      fp, fp, fp, fp, fp, vp, sz, vp]
    lib.resonator_state_init.restype = i32
    lib.resonator_state_init.argtypes = [vp, i32, i64, i64, i64, i64, fp, fp, fp, fp, fp, vp, sz, vp]
    lib.resonator_set_kernel_timer.restype = i32
    lib.resonator_set_kernel_timer.argtypes = [vp, vp]
    f32 = ctypes.c_float
    lib.resonator_epilogue_fwd.restype = i32
    lib.resonator_epilogue_fwd.argtypes = [vp, vp, vp, i32, vp, i64, i64, i64, i64, i64, fp, f32, fp, fp, vp]
    lib.resonator_epilogue_proj_fwd.restype = i32
    lib.resonator_epilogue_proj_fwd.argtypes = [vp, vp, vp, i32, vp, vp, vp, i64, i64, i64, i64, i64, i64, fp, f32, fp,
                                                fp, vp]
    lib.resonator_epilogue_workspace_bytes.restype = sz
    lib.resonator_epilogue_workspace_bytes.argtypes = [i64, i64, i64, i64, i64]
    lib.resonator_epilogue_bwd.restype = i32
    lib.resonator_epilogue_bwd.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp, i64, i64, i64, i64, i64, fp, f32,
                                           fp, fp, fp, fp, fp, fp, vp, sz, vp]
    lib.resonator_decode_step.restype = i32
    lib.resonator_decode_step.argtypes = [vp, i32, vp, i32, i64, i64, i64, fp, fp, fp, fp, fp, vp]
    lib.resonator_diagnostics.restype = i32
    lib.resonator_diagnostics.argtypes = [fp, fp, fp, fp, i64, i64, i64, fp, fp, fp, vp]
    lib.resonator_params_map.restype = i32
    lib.resonator_params_map.argtypes = [fp, fp, i64, f32, fp, fp, vp]
    lib.resonator_params_map_bwd.restype = i32
    lib.resonator_params_map_bwd.argtypes = [fp, fp, fp, fp, i64, fp, fp, vp]
    lib.resonator_params_init.restype = i32
    lib.resonator_params_init.argtypes = [i64, i64, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                          ctypes.c_double, f32, fp, fp, vp]
    lib.resonator_quadratic_reference_workspace_bytes.restype = sz
    lib.resonator_quadratic_reference_workspace_bytes.argtypes = [i64, i64]
    lib.resonator_quadratic_reference.restype = i32
    lib.resonator_quadratic_reference.argtypes = [vp, vp, i64, i64, i64, i64, fp, fp, fp, fp, vp, sz, vp]
    lib.resonator_fft_reference_workspace_bytes.restype = sz
    lib.resonator_fft_reference_workspace_bytes.argtypes = [i64, i64, i64]
    lib.resonator_fft_reference.restype = i32
    lib.resonator_fft_reference.argtypes = [vp, vp, i64, i64, i64, i64, fp, fp, fp, fp, vp, sz, vp]
    lib.resonator_grouped_linear.restype = i32
    lib.resonator_grouped_linear.argtypes = [vp, vp, i32, vp, i64, i64, i64, i64, vp]
    lib.resonator_grouped_linear2.restype = i32
    lib.resonator_grouped_linear2.argtypes = [vp, vp, vp, i32, vp, vp, i64, i64, i64, i64, vp]
    lib.resonator_block_diag_weight.restype = i32
    lib.resonator_block_diag_weight.argtypes = [vp, i32, i64, i64, i64, vp, vp]
    lib.resonator_block_diag_extract.restype = i32
    lib.resonator_block_diag_extract.argtypes = [fp, i64, i64, i64, fp, i32, vp]
    lib.resonator_grouped_linear_bwd_data.restype = i32
    lib.resonator_grouped_linear_bwd_data.argtypes = [vp, vp, i32, vp, i64, i64, i64, i64, i32, vp]
    lib.resonator_grouped_linear_bwd_data_sum.restype = i32
    lib.resonator_grouped_linear_bwd_data_sum.argtypes = [i32, ctypes.POINTER(vp), ctypes.POINTER(vp), i32, vp, i64, i64,
                                                          i64, i64, i32, vp]
    lib.resonator_grouped_linear_bwd_weight_sum_workspace_bytes.restype = sz
    lib.resonator_grouped_linear_bwd_weight_sum_workspace_bytes.argtypes = [i32, i32, i64, i64, i64, i64, i32]
    lib.resonator_grouped_linear_bwd_weight_sum.restype = i32
    lib.resonator_grouped_linear_bwd_weight_sum.argtypes = [i32, vp, ctypes.POINTER(vp), ctypes.POINTER(i32), i32, fp,
                                                            fp, i64, i64, i64, i64, i32, vp, sz, vp]
    lib.resonator_grouped_linear_bwd_weight.restype = i32
    lib.resonator_grouped_linear_bwd_weight.argtypes = [vp, vp, i32, fp, i64, i64, i64, i64, i32, vp]
    lib.resonator_grouped_linear_bwd_weight_split_workspace_bytes.restype = sz
    lib.resonator_grouped_linear_bwd_weight_split_workspace_bytes.argtypes = [i64, i64, i64]
    lib.resonator_grouped_linear_bwd_weight_split.restype = i32
    lib.resonator_grouped_linear_bwd_weight_split.argtypes = [vp, vp, i32, fp, i64, i64, i64, i64, i32, vp, sz, vp]
    lib.resonator_mix_fwd_noalloc.restype = i32
    lib.resonator_mix_fwd_noalloc.argtypes = [vp, i32, vp, i32, i64, i64, i64, i64, fp, fp, fp, fp, fp, fp, vp]
    lib.resonator_fwd_status.restype = i32
    lib.resonator_fwd_status.argtypes = [vp, ctypes.POINTER(ctypes.c_uint32), vp]
    lib.resonator_fwd_status_noalloc.restype = i32
    lib.resonator_fwd_status_noalloc.argtypes = [ctypes.POINTER(ctypes.c_uint32), vp]
    lib.resonator_mix_fwd_noalloc_max_bytes.restype = sz
    lib.resonator_mix_fwd_noalloc_max_bytes.argtypes = []
    lib.resonator_decode_steps.restype = i32
    lib.resonator_decode_steps.argtypes = [vp, i32, vp, i32, i64, i64, i64, i64, fp, fp, fp, fp, fp, vp]
    lib.resonator_decode_constants.restype = i32
    lib.resonator_decode_constants.argtypes = [i64, i64, fp, fp, fp, fp, fp, vp]
    lib.resonator_decode_step_tab.restype = i32
    lib.resonator_decode_step_tab.argtypes = [vp, i32, vp, i32, i64, i64, i64, fp, fp, vp]


def lib():
    """The loaded library (loaded once).  Raises if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() first "
                               "(there is no CPU or PyTorch fallback)")
        l = ctypes.CDLL(LIB_PATH)
        _declare(l)
        _lib = l
    return _lib


def check(rc: int):
    if rc != RES_OK:
        raise ResonatorError(rc, lib().resonator_last_error().decode(errors="replace"))
