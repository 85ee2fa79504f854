"""ctypes loader for libfastbfp.so (the C ABI of include/fastbfp.h).

There is no fallback: if the built library is missing or does not export the
ABI, importing the binding's entry points raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfastbfp.so")

# Every symbol the header declares, with its ctypes signature.
_P = ctypes.c_void_p
_I = ctypes.c_int
_I64 = ctypes.c_int64
_U64 = ctypes.c_uint64
SIGNATURES = {
    "bfp_abi_version": (_I, []),
    "bfp_status_str": (ctypes.c_char_p, [_I]),
    "bfp_chunks": (_I, [_I]),
    "bfp_quantized_sizes": (_I, [_I64, _I64, _I, _I, ctypes.POINTER(ctypes.c_size_t),
                                 ctypes.POINTER(ctypes.c_size_t)]),
    "bfp_quantize": (_I, [_P, _I64, _I64, _I, _I, _I, _I, _U64, _P, _P, _P, _P]),
    "bfp_quantize_nd": (_I, [_P, _I, _P, _I, _I, _I, _I, _U64, _P, _P, _P, _P]),
    "bfp_dequantize": (_I, [_P, _P, _I64, _I64, _I, _I, _P, _P]),
    "bfp_gemm": (_I, [_P, _P, _I, _P, _P, _I, _I64, _I64, _I64, _I, _I, _I, _P, _I64, _P]),
    "bfp_gemm_tiled": (_I, [_P, _P, _I, _P, _P, _I, _I64, _I64, _I64, _I, _I, _I, _P, _I64, _I, _P]),
    "bfp_gemm_group_partials": (_I, [_P, _I, _P, _I, _I64, _I64, _I64, _I, _I, _I, _P, _P]),
    "bfp_gemm_bfp": (_I, [_P, _P, _I, _P, _P, _I, _I64, _I64, _I64, _I, _I, _I, _I, _I, _U64, _P, _P, _P, _P]),
    "bfp_packed_sizes": (_I, [_I64, _I64, _I, ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)]),
    "bfp_quantize_packed": (_I, [_P, _I64, _I64, _I, _I, _U64, _P, _P, _P, _P]),
    "bfp_dequantize_packed": (_I, [_P, _P, _I64, _I64, _I, _P, _P]),
    "bfp_gemm_packed": (_I, [_P, _P, _I, _P, _P, _I, _I64, _I64, _I64, _I, _I, _P, _I64, _P]),
    "bfp_repack_sizes": (_I, [_I64, _I64, _I, _I, ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t),
                              ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int)]),
    "bfp_repack": (_I, [_P, _P, _I64, _I64, _I, _I, _I, _I, _P, _P, _P]),
    "bfp_gemm_ws_size": (_I, [_I, _I, _I64, _I64, _I64, _I, _I, _I, _I, ctypes.POINTER(ctypes.c_size_t)]),
    "bfp_gemm_ws": (_I, [_P, _P, _I, _P, _P, _I, _I64, _I64, _I64, _I, _I, _I, _I, _P, _I64, _P, ctypes.c_size_t, _P]),
    "bfp_quantize_dual": (_I, [_P, _I64, _I64, _I, _I, _I, _U64, _U64, _P, _P, _P, _P, _P, _P]),
    "bfp_weight_update": (_I, [_P, _P, ctypes.c_float, _P, _I64, _I64, _I, _I, _I, _U64, _U64, _P, _P, _P, _P, _P,
                               _P]),
    "bfp_quantize_adaptive": (_I, [_P, _I64, _I64, _I, _I, _I, _U64, _P, _P, _P, _P, _P, _P]),
    "bfp_adaptive_sums_len": (_I64, [_I64, _I64, _I, _I]),
    "bfp_quantize_adaptive_noalloc": (_I, [_P, _I64, _I64, _I, _I, _I, _U64, _P, _P, _P, _P, _P, _P]),
    "bfp_adaptive_parts": (_I64, [_I64, _I64, _I, _I]),
    "bfp_adaptive_noalloc_max_parts": (_I64, []),
    "bfp_adaptive_threshold": (ctypes.c_double, [ctypes.c_double, ctypes.c_double, _I64, _I64, _I64, _I64]),
    "bfp_adaptive_mantissa": (_I, [ctypes.c_double, ctypes.c_double, ctypes.c_double]),
}
ABI_VERSION = 7

_lock = threading.Lock()
_lib = None


class BFPError(RuntimeError):
    """A non-zero bfp_status_t returned by the library."""

    def __init__(self, status: int, where: str, message: str):
        super().__init__("%s failed with status %d: %s" % (where, status, message))
        self.status = status


def load() -> ctypes.CDLL:
    """Load libfastbfp.so once; raise if it is absent or incompatible."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError("libfastbfp.so is not built (%s); run paper_2110_15456_amd.build.build()" % LIB_PATH)
            lib = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            if lib.bfp_abi_version() != ABI_VERSION:
                raise ImportError("libfastbfp.so ABI %d, binding expects %d" % (lib.bfp_abi_version(), ABI_VERSION))
            _lib = lib
    return _lib


def check(status: int, where: str) -> None:
    if status != 0:
        raise BFPError(status, where, load().bfp_status_str(status).decode())
