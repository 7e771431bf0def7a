"""ctypes loader for libstarquant.so.  Raises if the library has not been built;
there is no fallback implementation."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libstarquant.so")

SQ_OK, SQ_ERR_NULL, SQ_ERR_SHAPE, SQ_ERR_ALIGN, SQ_ERR_WORKSPACE, SQ_ERR_HIP = range(6)

# name -> (restype, argtypes); mirrors include/starquant.h
_p, _i32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
SIGNATURES = {
    "sq_last_error": (ctypes.c_char_p, []),
    "sq_version": (ctypes.c_char_p, []),
    "sq_tac_default_block": (_i32, [_i32]),
    "sq_quant_act_workspace_bytes": (_sz, [_i32, _i32, _i32, _i32]),
    "sq_prepare_weights_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "sq_gemm_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "sq_gemm_w8_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "sgat_prepare_weights": (ctypes.c_int, [_p, _p, _i32, _i32, _p, _p, _p, _sz, _p]),
    "sgat_transform": (ctypes.c_int, [_p, _p, _p, _i32, _i32, _i32, _i32, _p, _p]),
    "sgat_quantize": (ctypes.c_int, [_p, _i32, _i32, _p, _p, _p]),
    "sgat_quant_act": (ctypes.c_int, [_p, _p, _p, _i32, _i32, _i32, _i32, _p, _p, _i32, _p, _p, _p, _sz, _p]),
    "w4a4_gemm": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _p, _p, _p, _sz, _p]),
    "tac_apply": (ctypes.c_int, [_p, _p, _p, _i32, _i32, _i32, _p, _p]),
    "sgat_prepare_weights_w8": (ctypes.c_int, [_p, _p, _i32, _i32, _p, _p, _p, _sz, _p]),
    "sgat_quantize_w8": (ctypes.c_int, [_p, _i32, _i32, _p, _p, _p]),
    "sgat_quant_act_w8": (ctypes.c_int, [_p, _p, _p, _i32, _i32, _i32, _i32, _p, _p, _i32, _p, _p, _p, _sz, _p]),
    "w8a8_gemm": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _p, _p, _p, _sz, _p]),
    "sgat_split_basis": (ctypes.c_int, [_p, _i32, _p, _p]),
    "sgat_transform_fast": (ctypes.c_int, [_p, _p, _p, _i32, _i32, _i32, _i32, _p, _p]),
    "sq_fp6_row_bytes": (_sz, [_i32]),
    "sq_codes_to_fp6": (ctypes.c_int, [_p, _i32, _i32, _p, _p]),
    "w4a4_gemm_fp6": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _p, _p, _p]),
    "sq_frag_weight_bytes": (_sz, [_i32, _i32]),
    "sq_weights_to_frag": (ctypes.c_int, [_p, _i32, _i32, _p, _p]),
    "w4a4_gemm_frag": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _p, _p, _p, _sz, _p]),
    "w4a4_gemm_frag_noalloc": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _p, _p, _p]),
    "sq_frag_weight_w8_bytes": (_sz, [_i32, _i32]),
    "sq_weights_to_frag_w8": (ctypes.c_int, [_p, _i32, _i32, _p, _p]),
    "w8a8_gemm_frag": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _p, _p, _p, _sz, _p]),
    "sq_tac_calibrate_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "tac_calibrate": (ctypes.c_int, [_p, _p, _i32, _i32, _i32, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_double, _p, _p, _p, _p, _p, _sz, _p]),
}


class StarQuantError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"starquant error {code}: {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2606_04945_amd.build` "
                "(there is no non-HIP implementation)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(rc: int) -> None:
    if rc != SQ_OK:
        raise StarQuantError(rc, lib().sq_last_error().decode())
