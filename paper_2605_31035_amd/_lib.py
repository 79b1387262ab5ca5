"""ctypes handle on libmixfp4.so with the C ABI's argument types.

Loading fails loudly: there is no pure-Python or CPU implementation of the
path behind this handle.  torch must be imported first so that the library
binds to the HIP runtime torch already loaded (same soname).
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (loads the HIP runtime the library binds to)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmixfp4.so")

SYMBOLS = ("mixfp4_quantize", "mixfp4_quantize_ex", "mixfp4_quantize_2d", "mixfp4_hadamard",
           "mixfp4_dequantize",
           "mixfp4_gemm", "mixfp4_gemm_ws", "mixfp4_gemm_workspace_size",
           "mixfp4_decode_operand", "mixfp4_gemm_decoded", "mixfp4_gemm_noalloc",
           "mixfp4_gemm_noalloc_max_bytes", "mixfp4_decode_step",
           "mixfp4_quantize_variant", "mixfp4_dequantize_variant", "mixfp4_quantize_decode",
           "mixfp4_status_string", "mixfp4_last_launch_error", "mixfp4_abi_version")


class MixFP4Error(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} not found: build it with `python paper_2605_31035_amd/build.py`")
    h = ctypes.CDLL(path)
    vp, i64, u32, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint, ctypes.c_int
    h.mixfp4_quantize.argtypes = [vp, i64, i64, i64, vp, vp, vp, u32, vp]
    h.mixfp4_quantize.restype = i32
    u64 = ctypes.c_uint64
    h.mixfp4_quantize_ex.argtypes = [vp, i64, i64, i64, vp, vp, vp, u32, i32, vp, u64, u64, vp]
    h.mixfp4_quantize_ex.restype = i32
    h.mixfp4_quantize_2d.argtypes = [vp, i64, i64, i64, vp, vp, vp, vp, vp, u32, vp]
    h.mixfp4_quantize_2d.restype = i32
    h.mixfp4_hadamard.argtypes = [vp, i64, i64, i64, i32, vp, vp, vp]
    h.mixfp4_hadamard.restype = i32
    h.mixfp4_dequantize.argtypes = [vp, vp, vp, i64, i64, vp, vp]
    h.mixfp4_dequantize.restype = i32
    h.mixfp4_gemm.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, vp, vp]
    h.mixfp4_gemm.restype = i32
    h.mixfp4_gemm_ws.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, vp, vp, i64, vp]
    h.mixfp4_gemm_ws.restype = i32
    h.mixfp4_gemm_workspace_size.argtypes = [i64, i64, i64, ctypes.POINTER(i64)]
    h.mixfp4_gemm_workspace_size.restype = i32
    h.mixfp4_decode_operand.argtypes = [vp, vp, i64, i64, vp, i64, ctypes.POINTER(i64), vp]
    h.mixfp4_decode_operand.restype = i32
    h.mixfp4_gemm_decoded.argtypes = [vp, vp, vp, vp, i64, i64, i64, vp, vp]
    h.mixfp4_gemm_decoded.restype = i32
    h.mixfp4_gemm_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, vp, vp]
    h.mixfp4_gemm_noalloc.restype = i32
    h.mixfp4_decode_step.argtypes = [vp, i64, i64, vp, vp, vp, i64, vp, vp, vp, vp, vp, vp]
    h.mixfp4_decode_step.restype = i32
    h.mixfp4_quantize_variant.argtypes = [vp, i64, i64, i64, i32, u32, vp, vp, vp, vp, u32, vp]
    h.mixfp4_quantize_variant.restype = i32
    h.mixfp4_dequantize_variant.argtypes = [vp, vp, vp, vp, i64, i64, i32, u32, vp, vp]
    h.mixfp4_dequantize_variant.restype = i32
    h.mixfp4_quantize_decode.argtypes = [vp, i64, i64, i64, vp, vp, vp, vp, i64, u32, vp]
    h.mixfp4_quantize_decode.restype = i32
    h.mixfp4_gemm_noalloc_max_bytes.argtypes = []
    h.mixfp4_gemm_noalloc_max_bytes.restype = i64
    h.mixfp4_status_string.argtypes = [i32]
    h.mixfp4_status_string.restype = ctypes.c_char_p
    h.mixfp4_last_launch_error.argtypes = []
    h.mixfp4_last_launch_error.restype = ctypes.c_char_p
    h.mixfp4_abi_version.argtypes = []
    h.mixfp4_abi_version.restype = i32
    return h


lib = load()
