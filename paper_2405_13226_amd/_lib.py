"""ctypes loader for ``libdd_attn.so`` (the C ABI of include/dd_attn.h).

The library is built in-tree by ``paper_2405_13226_amd.build``.  There is no
fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdd_attn.so")

# name -> (restype, argtypes); mirrors include/dd_attn.h
_P, _I, _F = ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p
SIGNATURES = {
    "dd_attn_fwd": (ctypes.c_int, [_P, _P, _P, _P, _F, _I, _I, _I, _I, _I, _P, _I, _P]),
    "dd_attn_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _F, _P, _P, _P, _I, _I, _I, _I, _I,
                                   _P, _I, _P, ctypes.c_size_t, _P]),
    "dd_attn_bwd_workspace_bytes": (ctypes.c_size_t, [_I, _I, _I, _I]),
    "dd_doclens_check": (ctypes.c_int, [_P, _I, ctypes.c_longlong]),
    "dd_status_str": (ctypes.c_char_p, [_I]),
}

STATUS = {
    0: "DD_OK", 1: "DD_ERR_NULL", 2: "DD_ERR_SHAPE", 3: "DD_ERR_HEADDIM",
    4: "DD_ERR_DOCLENS", 5: "DD_ERR_WORKSPACE", 6: "DD_ERR_ALIGN", 7: "DD_ERR_ALIAS",
    8: "DD_ERR_HIP",
}

_lib = None


class LibraryMissing(RuntimeError):
    pass


def lib():
    """The loaded library (raises LibraryMissing if it was never built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise LibraryMissing(
                f"{LIB_PATH} not found: build it with `python -m paper_2405_13226_amd.build`")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


class DDError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = lib().dd_status_str(status).decode()
        super().__init__(f"{where}: {STATUS.get(status, status)} ({msg})")


def check(status: int, where: str) -> None:
    if status != 0:
        raise DDError(status, where)
