"""Python binding of the block kernels around the attention (argument
marshalling only): the bf16 GEMM, LayerNorm and SwiGLU of include/dd_attn.h.

Every computation runs in the HIP kernels behind the C ABI; this module
checks tensor metadata, allocates outputs and scratch with torch on the
tensors' device and passes raw pointers, strides and the current stream.
Matrices are 2-D bf16 tensors with unit column stride (row-major, possibly
a column slice of a wider matrix: the row stride is passed through).
"""
from __future__ import annotations

import ctypes

import torch

from ._lib import check, lib

LN_EPS = 1e-5


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(dev):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _mat(t, name):
    if not isinstance(t, torch.Tensor) or t.dim() != 2:
        raise ValueError(f"{name} must be a 2-D tensor")
    if t.device.type != "cuda" or t.dtype != torch.bfloat16:
        raise ValueError(f"{name} must be a bf16 GPU tensor")
    if t.stride(1) != 1:
        raise ValueError(f"{name} must have unit column stride")


def gemm(a, b, trans_a: bool = False, trans_b: bool = False, residual=None, out=None):
    """op(a) @ op(b) (+ residual) in bf16 with fp32 accumulation.

    op(a) = a, or a.T when ``trans_a`` (a stored [K, M]); op(b) likewise.
    ``out`` (optional) receives the result and may be ``residual`` itself."""
    _mat(a, "a")
    _mat(b, "b")
    M, K = (a.shape[1], a.shape[0]) if trans_a else (a.shape[0], a.shape[1])
    Kb, N = (b.shape[1], b.shape[0]) if trans_b else (b.shape[0], b.shape[1])
    if K != Kb:
        raise ValueError(f"inner dimensions differ: {K} vs {Kb}")
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    _mat(out, "out")
    if tuple(out.shape) != (M, N):
        raise ValueError(f"out has shape {tuple(out.shape)}, expected {(M, N)}")
    if residual is not None:
        _mat(residual, "residual")
        if tuple(residual.shape) != (M, N) or residual.stride(0) != out.stride(0):
            raise ValueError("residual must match out in shape and row stride")
    need = lib().dd_gemm_workspace_bytes(M, N, K)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=a.device) if need else None
    st = lib().dd_gemm(_p(a), a.stride(0), int(bool(trans_a)), _p(b), b.stride(0),
                       int(bool(trans_b)), _p(residual), _p(out), out.stride(0), M, N, K,
                       _p(ws), need, _stream(a.device))
    check(st, "dd_gemm")
    return out


def transpose(x, out=None):
    """x.T as a bf16 matrix with unit column stride (into ``out`` if given)."""
    _mat(x, "x")
    R, C = x.shape
    if out is None:
        out = torch.empty((C, R), dtype=torch.bfloat16, device=x.device)
    _mat(out, "out")
    if tuple(out.shape) != (C, R):
        raise ValueError(f"out has shape {tuple(out.shape)}, expected {(C, R)}")
    st = lib().dd_transpose(_p(x), x.stride(0), _p(out), out.stride(0), R, C,
                            _stream(x.device))
    check(st, "dd_transpose")
    return out


def layer_norm(x, w, b, eps: float = LN_EPS):
    """(y, mean, rstd) of LayerNorm over the rows of x [rows, d]."""
    _mat(x, "x")
    rows, d = x.shape
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    y = torch.empty_like(x)
    mean = torch.empty(rows, dtype=torch.float32, device=x.device)
    rstd = torch.empty(rows, dtype=torch.float32, device=x.device)
    st = lib().dd_layernorm_fwd(_p(x), _p(w), _p(b), _p(y), _p(mean), _p(rstd), rows, d,
                                float(eps), _stream(x.device))
    check(st, "dd_layernorm_fwd")
    return y, mean, rstd


def layer_norm_backward(x, w, mean, rstd, dy, dres=None):
    """(dx, dw, db) of LayerNorm; ``dres`` (optional) is added to dx."""
    rows, d = x.shape
    dx = torch.empty_like(x)
    dw = torch.empty(d, dtype=torch.bfloat16, device=x.device)
    db = torch.empty(d, dtype=torch.bfloat16, device=x.device)
    need = lib().dd_layernorm_bwd_workspace_bytes(rows, d)
    ws = torch.empty(max(need, 16), dtype=torch.uint8, device=x.device)
    st = lib().dd_layernorm_bwd(_p(x), _p(w), _p(mean), _p(rstd), _p(dy.contiguous()),
                                _p(dres), _p(dx), _p(dw), _p(db), rows, d, _p(ws), ws.numel(),
                                _stream(x.device))
    check(st, "dd_layernorm_bwd")
    return dx, dw, db


def swiglu(u, v):
    """silu(u) * v elementwise."""
    y = torch.empty_like(u)
    st = lib().dd_swiglu_fwd(_p(u), _p(v), _p(y), u.numel(), _stream(u.device))
    check(st, "dd_swiglu_fwd")
    return y


def swiglu_backward(u, v, dy):
    """(du, dv) of y = silu(u) * v."""
    du, dv = torch.empty_like(u), torch.empty_like(v)
    st = lib().dd_swiglu_bwd(_p(u), _p(v), _p(dy.contiguous()), _p(du), _p(dv), u.numel(),
                             _stream(u.device))
    check(st, "dd_swiglu_bwd")
    return du, dv
