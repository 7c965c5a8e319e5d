"""ctypes loader for ``libcatekv.so`` (the C ABI declared in include/catekv.h)."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcatekv.so")

c_int, c_i64, c_size, c_void_p, c_double, c_float = (
    ctypes.c_int, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_double, ctypes.c_float)
P_i32 = ctypes.POINTER(ctypes.c_int32)
P_i64 = ctypes.POINTER(ctypes.c_int64)
P_f32 = ctypes.POINTER(ctypes.c_float)
P_u8 = ctypes.POINTER(ctypes.c_uint8)

CATEKV_OK = 0
CATEKV_ERR_INVALID_ARG = -1
CATEKV_ERR_UNSUPPORTED = -2
CATEKV_ERR_WORKSPACE = -3
CATEKV_ERR_HIP = -4
CATEKV_F32 = 0
CATEKV_BF16 = 1


class DecodePlanT(ctypes.Structure):
    _fields_ = [
        ("magic", ctypes.c_uint64),
        ("batch", ctypes.c_int32), ("hq", ctypes.c_int32), ("hkv", ctypes.c_int32),
        ("split_tokens", ctypes.c_int32),
        ("n_workers", ctypes.c_int32), ("n_segments", ctypes.c_int32), ("n_slots", ctypes.c_int32),
        ("n_multi", ctypes.c_int32),
        ("variant", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("segs_off", ctypes.c_uint64), ("workers_off", ctypes.c_uint64), ("views_off", ctypes.c_uint64),
        ("slots_off", ctypes.c_uint64),
        ("ws_bytes", ctypes.c_uint64),
        ("max_len_total", ctypes.c_int64),
    ]


# name -> (restype, argtypes)
SIGNATURES = {
    "catekv_score_heads_workspace": (c_size, [c_int, c_int, c_int, c_i64, c_i64, c_i64]),
    "catekv_score_heads": (c_int, [c_int, c_void_p, c_i64, c_void_p, c_int, c_int, c_int, c_i64, c_int,
                                   c_i64, c_i64, c_double, c_double, c_int, c_void_p, c_void_p, c_size,
                                   c_void_p]),
    "catekv_classify_heads": (c_int, [P_f32, c_int, c_int, c_double, P_u8]),
    "catekv_adaptive_budget": (c_int, [c_i64, c_int, c_int, c_double, P_i64]),
    "catekv_select_workspace": (c_size, [c_int, c_int, c_int, c_i64, c_int, c_int]),
    "catekv_select_critical": (c_int, [c_int, c_void_p, c_void_p, c_int, c_int, c_int, c_i64, c_int, c_int,
                                       P_i32, c_int, c_int, c_void_p, c_void_p, c_size, c_void_p]),
    "catekv_select_critical_noalloc": (c_int, [c_int, c_void_p, c_void_p, c_int, c_int, c_int, c_i64, c_int, c_int,
                                               P_i32, c_int, c_int, c_void_p, c_void_p]),
    "catekv_compact_kv": (c_int, [c_int, c_void_p, c_void_p, c_int, c_i64, c_int, c_int, c_int, P_i32, c_int,
                                  c_void_p, c_int, c_void_p, c_void_p, c_void_p, c_void_p]),
    "catekv_decode_workspace": (c_size, [P_i64, c_int, c_int, c_int, c_int]),
    "catekv_decode_plan": (c_int, [P_i64, c_int, c_int, c_int, c_int, ctypes.POINTER(DecodePlanT), c_void_p,
                                   c_size, c_void_p]),
    "catekv_decode_attn": (c_int, [c_int, ctypes.POINTER(DecodePlanT), c_void_p, c_void_p, c_void_p, c_int,
                                   c_int, c_int, c_int, c_float, c_void_p, c_void_p, c_void_p, c_size,
                                   c_void_p]),
    "catekv_page_bounds": (c_int, [c_int, c_void_p, c_int, c_i64, c_int, c_int, P_i32, c_int, c_void_p, c_void_p,
                                   c_void_p]),
    "catekv_retrieve_workspace": (c_size, [c_int, c_i64]),
    "catekv_retrieve_pages": (c_int, [c_int, c_void_p, c_void_p, c_void_p, c_int, c_int, c_i64, c_int, P_i32, c_int,
                                      c_int, c_void_p, c_void_p, c_size, c_void_p]),
    "catekv_append_kv": (c_int, [c_int, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_int, c_int, c_int,
                                 c_void_p, c_void_p]),
    "catekv_last_error": (ctypes.c_char_p, []),
    "catekv_version": (ctypes.c_char_p, []),
}

_lib = None


class CateKVError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"catekv status {status}: {msg}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library.  Raises if it has not been built: there is no
    fallback implementation."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2608_30295_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != CATEKV_OK:
        raise CateKVError(status, lib().catekv_last_error().decode())
