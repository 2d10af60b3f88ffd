"""ctypes binding of librcllm.so, the HIP (gfx950) selective-prefill library.

Argument marshalling only: every step of the path runs in the library's HIP
kernels. torch is imported first so that the library binds to the HIP runtime
torch already loaded (one runtime per process, so torch's stream handles are
valid in the library).
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (loads the HIP runtime the library must share)

PKG = os.path.dirname(os.path.abspath(__file__))
# RCLLM_LIB names another build of the library (e.g. one whose host code is
# built with AddressSanitizer); default: the in-tree build
LIB_PATH = os.environ.get("RCLLM_LIB") or os.path.join(PKG, "librcllm.so")

RC_OK, RC_ERR_INVALID_ARG, RC_ERR_UNSUPPORTED, RC_ERR_HIP = 0, -1, -2, -3
RC_F32, RC_BF16 = 0, 1

# every symbol include/rcllm.h declares
EXPORTS = ("rc_rope_table", "rc_kv_assemble", "rc_rerope", "rc_select_tokens",
           "rc_selective_attention", "rc_selective_attention_lse", "rc_attention_mass",
           "rc_select_tokens_eq3", "rc_paged_attention", "rc_segments_with_window",
           "rc_kv_gather_tokens", "rc_gemm_bf16", "rc_rmsnorm", "rc_qkv_rope", "rc_silu_mul",
           "rc_gather_rows", "rc_kv_assemble_vref", "rc_select_tokens_vref",
           "rc_selective_attention_vref",
           "rc_status_string", "rc_last_error")


class RcShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("N", ctypes.c_int32), ("Hq", ctypes.c_int32),
                ("Hkv", ctypes.c_int32), ("D", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class RcPool(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("num_blocks", ctypes.c_int32), ("block_len", ctypes.c_int32)]


class RcError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_string(status)}: {msg}")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load the built library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; "
                           "g.build()'` or `python paper_2605_07443_amd/build.py` first")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, f32, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_double
    P = ctypes.POINTER
    L.rc_rope_table.argtypes = [i32, i32, f64, vp, vp]
    L.rc_kv_assemble.argtypes = [P(RcShape), P(RcPool), i32, vp, i32, vp, vp, vp, vp, i32, vp, vp, vp,
                                 vp]
    L.rc_rerope.argtypes = [P(RcShape), vp, vp, vp, vp, i32, vp]
    L.rc_select_tokens.argtypes = [P(RcShape), vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, i32, vp]
    L.rc_selective_attention.argtypes = [P(RcShape), vp, vp, i32, vp, vp, f32, vp, vp]
    L.rc_selective_attention_lse.argtypes = [P(RcShape), vp, vp, i32, vp, vp, f32, vp, vp, vp]
    L.rc_attention_mass.argtypes = [P(RcShape), vp, vp, vp, f32, vp, vp]
    L.rc_select_tokens_eq3.argtypes = [P(RcShape), vp, i32, i32, ctypes.c_uint32, f32, i32, i32,
                                       vp, vp, vp, vp, vp, vp, vp, vp, i32, vp]
    L.rc_paged_attention.argtypes = [P(RcShape), vp, vp, i32, P(RcPool), i32, vp, i32, vp, vp, vp,
                                     vp, i32, f32, vp, vp]
    L.rc_segments_with_window.argtypes = [vp, i32, i32, i32, i32, vp, i32, P(i32)]
    L.rc_kv_gather_tokens.argtypes = [P(RcShape), P(RcPool), i32, vp, vp, vp, vp, vp, i32, vp, vp,
                                      vp, i32, vp]
    i64 = ctypes.c_int64
    L.rc_gemm_bf16.argtypes = [i64, i32, i32, vp, vp, vp, vp, vp]
    L.rc_rmsnorm.argtypes = [i32, i32, vp, vp, f32, vp, vp]
    L.rc_qkv_rope.argtypes = [P(RcShape), vp, vp, i32, vp, vp, i32, vp, vp, vp, vp]
    L.rc_silu_mul.argtypes = [i64, i32, vp, vp, vp]
    L.rc_gather_rows.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp]
    L.rc_kv_assemble_vref.argtypes = L.rc_kv_assemble.argtypes
    L.rc_select_tokens_vref.argtypes = [P(RcShape), vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp,
                                        vp]
    L.rc_selective_attention_vref.argtypes = [P(RcShape), vp, vp, i32, vp, vp, f32, vp, vp]
    for name in EXPORTS:
        if name not in ("rc_status_string", "rc_last_error"):
            getattr(L, name).restype = ctypes.c_int
    L.rc_status_string.argtypes = [ctypes.c_int]
    L.rc_status_string.restype = ctypes.c_char_p
    L.rc_last_error.argtypes = []
    L.rc_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def status_string(status: int) -> str:
    return load().rc_status_string(status).decode()


def last_error() -> str:
    return load().rc_last_error().decode()


def check(status: int) -> None:
    if status != RC_OK:
        raise RcError(status, last_error())
