"""ctypes binding to libsteel.so (argument marshalling only).

Every step of the attention pass runs in the library's HIP kernels; this
module only checks tensors, allocates the output with torch and passes raw
device pointers and torch's current HIP stream.  If the library is missing it
raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsteel.so")

STEEL_OK = 0
STEEL_ERR_INVALID_ARGUMENT = 1
STEEL_ERR_UNSUPPORTED = 2
STEEL_ERR_HIP = 3

_lib = None


class SteelError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libsteel status {status}: {message}")
        self.status = status


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libsteel.so (built by ``paper_2607_09385_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_2607_09385_amd.build` "
            "(the HIP library is required; there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    c_int, c_void_p, c_float = ctypes.c_int, ctypes.c_void_p, ctypes.c_float
    lib.steel_attn_fwd.restype = c_int
    lib.steel_attn_fwd.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                   c_int, c_int, c_int, c_int, c_int, c_int, c_int,
                                   c_float, c_int, c_void_p]
    lib.steel_block_index.restype = c_int
    lib.steel_block_index.argtypes = [c_void_p, c_int, c_int, c_int, c_int, c_int, c_int,
                                      c_void_p, c_void_p, c_void_p, c_void_p]
    c_size_t = ctypes.c_size_t
    lib.steel_attn_workspace_bytes.restype = c_size_t
    lib.steel_attn_workspace_bytes.argtypes = [c_int] * 6
    lib.steel_attn_plan.restype = c_int
    lib.steel_attn_plan.argtypes = [c_void_p] + [c_int] * 7 + [c_void_p, c_size_t, c_void_p]
    lib.steel_attn_run.restype = c_int
    lib.steel_attn_run.argtypes = [c_void_p] * 4 + [c_int] * 7 + [c_float, c_int, c_void_p,
                                                                  c_size_t, c_void_p]
    lib.steel_attn_fwd_window.restype = c_int
    lib.steel_attn_fwd_window.argtypes = [c_void_p] * 4 + [c_int] * 7 + [c_float, c_int, c_int,
                                                                         c_int, c_void_p]
    lib.steel_attn_plan_window.restype = c_int
    lib.steel_attn_plan_window.argtypes = [c_int] * 9 + [c_void_p, c_size_t, c_void_p]
    lib.steel_topk_block_mask.restype = c_int
    lib.steel_topk_block_mask.argtypes = [c_void_p, c_void_p] + [c_int] * 10 + [c_void_p, c_void_p]
    lib.steel_attn_fwd_ex.restype = c_int
    lib.steel_attn_fwd_ex.argtypes = [c_void_p] * 6 + [c_int] * 7 + [c_float, c_int, c_int, c_int,
                                                                     c_void_p]
    lib.steel_attn_fwd_noalloc.restype = c_int
    lib.steel_attn_fwd_noalloc.argtypes = list(lib.steel_attn_fwd.argtypes)
    lib.steel_attn_merge.restype = c_int
    lib.steel_attn_merge.argtypes = [c_void_p, c_void_p, c_int, ctypes.c_longlong, c_int, c_void_p,
                                     c_void_p, c_void_p]
    lib.steel_mfma_peak.restype = c_int
    lib.steel_mfma_peak.argtypes = [c_void_p, c_int, c_int, c_int, c_void_p, c_void_p, c_void_p]
    lib.steel_valu_rate.restype = c_int
    lib.steel_valu_rate.argtypes = [c_int, c_void_p, c_int, c_int, c_int, c_void_p, c_void_p, c_void_p]
    lib.steel_mix_rate.restype = c_int
    lib.steel_mix_rate.argtypes = [c_int, c_int, c_void_p, c_int, c_void_p, c_int, c_int, c_void_p,
                                   c_void_p, c_void_p]
    lib.steel_lds_rate.restype = c_int
    lib.steel_lds_rate.argtypes = [c_int, c_int, c_int, c_int, c_void_p, c_void_p, c_void_p]
    lib.steel_copy_rate.restype = c_int
    lib.steel_copy_rate.argtypes = [c_void_p, c_size_t, c_int, c_int, c_int, c_void_p, c_void_p, c_void_p]
    lib.steel_last_error.restype = ctypes.c_char_p
    lib.steel_last_error.argtypes = []
    lib.steel_version.restype = ctypes.c_char_p
    lib.steel_version.argtypes = []
    _lib = lib
    return lib


def last_error() -> str:
    return load().steel_last_error().decode()


def version() -> str:
    return load().steel_version().decode()


def check(status: int) -> None:
    if status != STEEL_OK:
        raise SteelError(status, last_error())
