"""fp64 CPU oracle for the dataset-decomposition attention hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the HIP library ``paper_2405_13226_amd`` and never imports it.

Contents
* ``attn_fwd`` / ``attn_bwd``: ctypes front-ends of ``attn_oracle.c``, the
  plain masked-attention definition in double precision (Sec. 2.1 and 2.2 of
  arXiv 2405.13226 for the mask and batch shape; Appendix F for the causal
  contexts 0..l-1).
* ``metrics``: average sequence length, average context length (Appendix F,
  eq. avg_context) and the count of allowed (query, key) pairs.
* ``decompose``: the binary dataset decomposition of Sec. 2.1.
* ``layer``: one OpenLM transformer block (fp64 torch plus the attention
  oracle), forward and backward.
* ``rope``: rotary position embedding of queries and keys (Sec. 3,
  "Positional encoding") around the attention definition.

Every function is pinned by ``tests/test_oracle_*.py`` against closed forms,
brute force on tiny inputs, finite differences, invariants and the values
printed in Table "mixture" of the paper.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "attn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = True) -> str:
    """Compile ``attn_oracle.c`` with gcc (fp64, OpenMP).  Returns the path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared",
                        "-std=c11", "-Wall", "-o", tmp, _SRC, "-lm"],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or (os.path.getmtime(_LIB)
                                        < os.path.getmtime(_SRC)):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        for name, nin in (("oracle_attn_fwd_bf16", 3), ("oracle_attn_fwd_f64", 3),
                          ("oracle_attn_bwd_bf16", 4), ("oracle_attn_bwd_f64", 4)):
            fn = getattr(lib, name)
            nout = 2 if "fwd" in name else 3
            fn.argtypes = [P] * nin + [I] * 5 + [P, I, P, I] + [P] * nout
            fn.restype = I
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = I
        _lib = lib
    return _lib


def threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(_load().oracle_threads())


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _prep(x, kind):
    if kind == "bf16":
        return np.ascontiguousarray(x, dtype=np.uint16)
    return np.ascontiguousarray(x, dtype=np.float64)


def _kind_of(q):
    return "bf16" if np.asarray(q).dtype == np.uint16 else "f64"


def _bh_array(bh, B, H):
    if bh is None:
        bh = [(b, h) for b in range(B) for h in range(H)]
    return np.ascontiguousarray(np.asarray(bh, dtype=np.int32).reshape(-1, 2))


def _doc_array(cu_doclens):
    if cu_doclens is None:
        return None, 0
    cu = np.ascontiguousarray(np.asarray(cu_doclens, dtype=np.int32))
    return cu, int(cu.size - 1)


def attn_fwd(q, k, v, causal=True, cu_doclens=None, bh=None):
    """Oracle forward.

    q, k, v: [B, L, H, D] arrays, either uint16 bf16 bit patterns or float64.
    cu_doclens: optional int offsets (n_docs + 1) over the flattened B*L axis.
    bh: optional list of (b, h) pairs; default all pairs in (b, h) order.
    Returns (o [n_bh, L, D] float64, lse [n_bh, L] float64).
    """
    kind = _kind_of(q)
    q, k, v = (_prep(x, kind) for x in (q, k, v))
    B, L, H, D = q.shape
    assert k.shape == q.shape and v.shape == q.shape
    bha = _bh_array(bh, B, H)
    cu, nd = _doc_array(cu_doclens)
    o = np.zeros((bha.shape[0], L, D), dtype=np.float64)
    lse = np.zeros((bha.shape[0], L), dtype=np.float64)
    fn = _load().oracle_attn_fwd_bf16 if kind == "bf16" else _load().oracle_attn_fwd_f64
    rc = fn(_ptr(q), _ptr(k), _ptr(v), B, L, H, D, int(bool(causal)), _ptr(cu),
            nd, _ptr(bha), bha.shape[0], _ptr(o), _ptr(lse))
    if rc != 0:
        raise ValueError("oracle_attn_fwd: bad arguments")
    return o, lse


def attn_bwd(q, k, v, do, causal=True, cu_doclens=None, bh=None):
    """Oracle backward of sum(dO * O).  Returns (dq, dk, dv), each [n_bh, L, D]."""
    kind = _kind_of(q)
    q, k, v, do = (_prep(x, kind) for x in (q, k, v, do))
    B, L, H, D = q.shape
    bha = _bh_array(bh, B, H)
    cu, nd = _doc_array(cu_doclens)
    outs = [np.zeros((bha.shape[0], L, D), dtype=np.float64) for _ in range(3)]
    fn = _load().oracle_attn_bwd_bf16 if kind == "bf16" else _load().oracle_attn_bwd_f64
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(do), B, L, H, D, int(bool(causal)),
            _ptr(cu), nd, _ptr(bha), bha.shape[0], *(_ptr(x) for x in outs))
    if rc != 0:
        raise ValueError("oracle_attn_bwd: bad arguments")
    return tuple(outs)


def to_blhd(x, B, H, bh=None):
    """Scatter compact [n_bh, L, D] oracle output back into [B, L, H, D]."""
    x = np.asarray(x)
    n, L = x.shape[0], x.shape[1]
    tail = x.shape[2:]
    out = np.zeros((B, L, H) + tail, dtype=x.dtype)
    pairs = _bh_array(bh, B, H)
    for p in range(n):
        out[pairs[p, 0], :, pairs[p, 1]] = x[p]
    return out


from . import metrics, decompose, rope, layer  # noqa: E402,F401
