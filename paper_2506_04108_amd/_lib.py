"""ctypes declarations of libresa.so (the C ABI in include/resa.h).

Loading fails loudly when the library has not been built: there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libresa.so")

RESA_OK = 0
STATUS_NAMES = {0: "RESA_OK", 1: "RESA_ERR_INVALID_ARG", 2: "RESA_ERR_UNSUPPORTED",
                3: "RESA_ERR_WORKSPACE", 4: "RESA_ERR_CAPACITY", 5: "RESA_ERR_HIP"}


class ResaError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {message}")
        self.code = code


class KVCacheDesc(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("kmin", C.c_void_p), ("kmax", C.c_void_p),
                ("batch", C.c_int32), ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("capacity", C.c_int32), ("block_size", C.c_int32),
                ("block_table", C.c_void_p), ("num_pages", C.c_int32)]


class SelectParams(C.Structure):
    _fields_ = [("sparsity", C.c_double), ("min_blocks", C.c_int32), ("n_local", C.c_int32)]


_P = C.c_void_p
_I = C.c_int32
_Z = C.c_size_t
_F = C.c_float
_D = C.c_double
_CACHE = C.POINTER(KVCacheDesc)

# name -> (restype, argtypes); mirrors include/resa.h.
SIGNATURES = {
    "resa_version": (C.c_char_p, []),
    "resa_last_error": (C.c_char_p, []),
    "resa_num_selected": (_I, [_I, _D, _I, _I]),
    "resa_block_summarize": (C.c_int, [_CACHE, _P, _I, _I, _P]),
    "resa_append_kv": (C.c_int, [_CACHE, _P, _P, _P, _I, _P]),
    "resa_select_workspace_size": (_Z, [_I, _I, _I, _I]),
    "resa_select_blocks": (C.c_int, [_CACHE, _P, _I, _P, _I, C.POINTER(SelectParams), _P, _P, _I,
                                     _P, _P, _Z, _P]),
    "resa_append_select": (C.c_int, [_CACHE, _P, _P, _P, _I, _P, _I, C.POINTER(SelectParams), _P, _P,
                                     _I, _P, _P, _Z, _P]),
    "resa_select_stats_offset": (_Z, [_I, _I]),
    "resa_step_stats_offset": (_Z, [_I, _I]),
    "resa_decode_num_splits": (_I, [_I, _I, _I, _I]),
    "resa_decode_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I]),
    "resa_sparse_decode": (C.c_int, [_CACHE, _P, _I, _P, _P, _P, _I, _I, _F, _P, _P, _P, _Z, _P]),
    "resa_sparse_decode_noalloc": (C.c_int, [_CACHE, _P, _I, _P, _P, _P, _I, _I, _F, _P, _P, _P]),
    "resa_sparse_decode_noalloc_max_bytes": (_Z, []),
    "resa_step_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I, _I]),
    "resa_decode_step": (C.c_int, [_CACHE, _P, _P, _P, _I, _P, _I, C.POINTER(SelectParams), _P, _P, _I,
                                   _I, _F, _P, _P, _P, _Z, _P]),
    "resa_rectify_workspace_size": (_Z, [_I, _I, _I, _I, _I]),
    "resa_dense_rectify": (C.c_int, [_CACHE, _P, _P, _P, _I, _I, _P, _P, _I, _F, _P, _P, _I, _P,
                                     _Z, _P]),
    "resa_workspace_clear": (C.c_int, [_P, _Z, _P]),
    "resa_stream_read": (C.c_int, [_P, _Z, _P, C.c_uint32, _I, _P]),
}

_lib = None


def lib() -> C.CDLL:
    """The loaded library (loaded once). Raises if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2506_04108_amd.build`")
        h = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


def check(rc: int) -> None:
    if rc != RESA_OK:
        raise ResaError(rc, lib().resa_last_error().decode())
