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
    "dd_attn_fwd_rope": (ctypes.c_int, [_P, _P, _P, _P, _F, _P, _I, _I, _I, _I, _I, _P, _I,
                                        ctypes.c_float, _I, _P]),
    "dd_attn_bwd_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _P, _F, _P, _P, _P, _I, _I, _I, _I,
                                           _I, _P, _I, _P]),
    "dd_attn_bwd_rope": (ctypes.c_int, [_P, _P, _P, _P, _P, _F, _P, _P, _P, _I, _I, _I, _I, _I,
                                        _P, _I, ctypes.c_float, _I, _P, ctypes.c_size_t, _P]),
    "dd_rope": (ctypes.c_int, [_P, _P, _I, _I, _I, _I, ctypes.c_float, _I, _P, _I, _I, _P]),
    "dd_attn_bwd_workspace_bytes": (ctypes.c_size_t, [_I, _I, _I, _I]),
    "dd_gemm": (ctypes.c_int, [_P, ctypes.c_longlong, _I, _P, ctypes.c_longlong, _I, _P, _P,
                               ctypes.c_longlong, _I, _I, _I, _P, ctypes.c_size_t, _P]),
    "dd_gemm_workspace_bytes": (ctypes.c_size_t, [_I, _I, _I]),
    "dd_layernorm_fwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _I, _I, ctypes.c_float, _P]),
    "dd_layernorm_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _P,
                                        ctypes.c_size_t, _P]),
    "dd_layernorm_bwd_workspace_bytes": (ctypes.c_size_t, [_I, _I]),
    "dd_swiglu_fwd": (ctypes.c_int, [_P, _P, _P, ctypes.c_longlong, _P]),
    "dd_transpose": (ctypes.c_int, [_P, ctypes.c_longlong, _P, ctypes.c_longlong, _I, _I, _P]),
    "dd_swiglu_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, ctypes.c_longlong, _P]),
    "dd_doclens_check": (ctypes.c_int, [_P, _I, ctypes.c_longlong]),
    "dd_status_str": (ctypes.c_char_p, [_I]),
    "dd_prof_enable": (ctypes.c_int, [_I]),
    "dd_prof_read": (ctypes.c_int, [_I, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_longlong)]),
    "dd_prof_kernel_name": (ctypes.c_char_p, [_I]),
    "dd_prof_launches": (ctypes.c_int, [_P, _P, ctypes.c_longlong,
                                        ctypes.POINTER(ctypes.c_longlong)]),
}

KERNELS = {"forward": 0, "backward_short": 1, "backward_dkdv": 2, "backward_dq": 3, "rope": 4}


def prof_enable(on: bool) -> None:
    check(lib().dd_prof_enable(int(bool(on))), "dd_prof_enable")


def prof_read(kernel: int):
    """(total ms, launches) of one kernel since the last prof_enable(True)."""
    ms, n = ctypes.c_double(0.0), ctypes.c_longlong(0)
    check(lib().dd_prof_read(int(kernel), ctypes.byref(ms), ctypes.byref(n)), "dd_prof_read")
    return ms.value, n.value

def prof_launches():
    """[(kernel id, ms)] of every launch recorded since prof_enable(True), in
    launch order."""
    import numpy as np
    n = ctypes.c_longlong(0)
    check(lib().dd_prof_launches(None, None, 0, ctypes.byref(n)), "dd_prof_launches")
    kid = np.zeros(max(n.value, 1), dtype=np.int32)
    ms = np.zeros(max(n.value, 1), dtype=np.float64)
    check(lib().dd_prof_launches(kid.ctypes.data_as(ctypes.c_void_p),
                                 ms.ctypes.data_as(ctypes.c_void_p), n.value, ctypes.byref(n)),
          "dd_prof_launches")
    return list(zip(kid[:n.value].tolist(), ms[:n.value].tolist()))


STATUS = {
    0: "DD_OK", 1: "DD_ERR_NULL", 2: "DD_ERR_SHAPE", 3: "DD_ERR_HEADDIM",
    4: "DD_ERR_DOCLENS", 5: "DD_ERR_WORKSPACE", 6: "DD_ERR_ALIGN", 7: "DD_ERR_ALIAS",
    8: "DD_ERR_HIP", 9: "DD_ERR_SCRATCH",
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
