"""Python binding of the DD attention hot path: argument marshalling only.

Every step of the computation runs in the HIP kernels behind the C ABI; this
module checks tensor metadata, allocates outputs with torch on the tensors'
device and passes raw pointers and the current stream.

Tensors are bf16, contiguous, [B, L, H, D] on a ROCm device; LSE is fp32
[B, L, H].  ``cu_doclens`` (optional) holds n_docs + 1 document start offsets
over the flattened B*L axis (the document-masked concat-and-chunk baseline);
it may be a list, a numpy array or an int32 tensor.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from ._lib import check, lib


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(dev):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _check_tensor(t, name, shape=None, dtype=torch.bfloat16):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU device (got {t.device})")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _empty(t) -> bool:
    """B, L or H is 0: nothing to compute.  The C ABI takes each >= 1, so
    the wrappers return empty results without calling it."""
    return t.dim() == 4 and t.shape[0] * t.shape[1] * t.shape[2] == 0


class DocLens:
    """Validated document offsets: a host copy and an int32 device copy."""

    def __init__(self, cu_doclens, total_tokens: int, device):
        if isinstance(cu_doclens, torch.Tensor):
            host = cu_doclens.detach().to("cpu", torch.int64).numpy()
        else:
            host = np.asarray(cu_doclens, dtype=np.int64)
        if host.ndim != 1 or host.size < 2:
            raise ValueError("cu_doclens needs at least two offsets")
        if host.max() >= 2 ** 31:
            raise ValueError("cu_doclens offsets must fit int32")
        self.host = np.ascontiguousarray(host.astype(np.int32))
        self.n_docs = int(self.host.size - 1)
        check(lib().dd_doclens_check(self.host.ctypes.data_as(ctypes.c_void_p), self.n_docs,
                                     int(total_tokens)), "dd_doclens_check")
        if (isinstance(cu_doclens, torch.Tensor) and cu_doclens.device == device
                and cu_doclens.dtype == torch.int32 and cu_doclens.is_contiguous()):
            self.dev = cu_doclens
        else:
            self.dev = torch.from_numpy(self.host).to(device)


def _doclens(cu_doclens, B, L, device):
    if cu_doclens is None:
        return None
    if isinstance(cu_doclens, DocLens):
        return cu_doclens
    return DocLens(cu_doclens, B * L, device)


def forward(q, k, v, causal: bool = True, cu_doclens=None):
    """Attention forward.  Returns (o [B,L,H,D] bf16, lse [B,L,H] fp32)."""
    _check_tensor(q, "q")
    B, L, H, D = q.shape
    _check_tensor(k, "k", q.shape)
    _check_tensor(v, "v", q.shape)
    o = torch.empty_like(q)
    lse = torch.empty((B, L, H), dtype=torch.float32, device=q.device)
    if _empty(q):
        return o, lse
    docs = _doclens(cu_doclens, B, L, q.device)
    st = lib().dd_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, L, H, D,
                           int(bool(causal)), _ptr(docs.dev) if docs else None,
                           docs.n_docs if docs else 0, _stream(q.device))
    check(st, "dd_attn_fwd")
    return o, lse


def workspace_bytes(B, L, H, D) -> int:
    return int(lib().dd_attn_bwd_workspace_bytes(B, L, H, D))


def backward(q, k, v, o, lse, do, causal: bool = True, cu_doclens=None, workspace=None):
    """Attention backward of sum(do * o).  Returns (dq, dk, dv), bf16."""
    _check_tensor(q, "q")
    B, L, H, D = q.shape
    for t, n in ((k, "k"), (v, "v"), (o, "o"), (do, "do")):
        _check_tensor(t, n, q.shape)
    _check_tensor(lse, "lse", (B, L, H), torch.float32)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    if _empty(q):
        return dq, dk, dv
    docs = _doclens(cu_doclens, B, L, q.device)
    need = workspace_bytes(B, L, H, D)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    st = lib().dd_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse),
                           _ptr(dq), _ptr(dk), _ptr(dv), B, L, H, D, int(bool(causal)),
                           _ptr(docs.dev) if docs else None, docs.n_docs if docs else 0,
                           _ptr(workspace), workspace.numel() * workspace.element_size(),
                           _stream(q.device))
    check(st, "dd_attn_bwd")
    return dq, dk, dv


def rope(x, base: float, cu_doclens=None, doc_positions: bool = False, inverse: bool = False,
         out=None):
    """Rotary position embedding of a [B, L, H, D] bf16 tensor (new tensor, or
    ``out``, which may be ``x`` itself)."""
    _check_tensor(x, "x")
    B, L, H, D = x.shape
    y = torch.empty_like(x) if out is None else out
    if out is not None:
        _check_tensor(out, "out", x.shape)
    if _empty(x):
        return y
    docs = _doclens(cu_doclens, B, L, x.device)
    st = lib().dd_rope(_ptr(x), _ptr(y), B, L, H, D, float(base), int(bool(inverse)),
                       _ptr(docs.dev) if docs else None, docs.n_docs if docs else 0,
                       int(bool(doc_positions)), _stream(x.device))
    check(st, "dd_rope")
    return y


def forward_rope(q, k, v, base: float, causal: bool = True, cu_doclens=None,
                 doc_positions: bool = False, fused: bool = True):
    """Attention over rotated q and k.  Returns (o, lse, q_rot, k_rot); the
    rotated tensors are what ``backward_rope`` takes.  With ``fused`` the
    attention kernel rotates q as it loads it (and writes q_rot); otherwise
    q is rotated by a separate dd_rope pass.  k is always rotated by
    dd_rope.  Both give bit-identical results."""
    B, L = q.shape[0], q.shape[1]
    docs = None if _empty(q) else _doclens(cu_doclens, B, L, q.device)
    kr = rope(k, base, docs, doc_positions)
    if not fused or _empty(q):
        qr = rope(q, base, docs, doc_positions)
        o, lse = forward(qr, kr, v, causal, docs)
        return o, lse, qr, kr
    _check_tensor(q, "q")
    for t, n in ((kr, "k"), (v, "v")):
        _check_tensor(t, n, q.shape)
    H, D = q.shape[2], q.shape[3]
    qr = torch.empty_like(q)
    o = torch.empty_like(q)
    lse = torch.empty((B, L, H), dtype=torch.float32, device=q.device)
    st = lib().dd_attn_fwd_rope(_ptr(q), _ptr(kr), _ptr(v), _ptr(o), _ptr(lse), _ptr(qr),
                                B, L, H, D, int(bool(causal)),
                                _ptr(docs.dev) if docs else None, docs.n_docs if docs else 0,
                                float(base), int(bool(doc_positions)), _stream(q.device))
    check(st, "dd_attn_fwd_rope")
    return o, lse, qr, kr


def backward_rope(q_rot, k_rot, v, o, lse, do, base: float, causal: bool = True,
                  cu_doclens=None, doc_positions: bool = False, workspace=None):
    """Backward of attention over rotated q, k: (dq, dk, dv) with respect to
    the unrotated q and k (the kernels rotate the gradients back)."""
    _check_tensor(q_rot, "q_rot")
    B, L, H, D = q_rot.shape
    for t, n in ((k_rot, "k_rot"), (v, "v"), (o, "o"), (do, "do")):
        _check_tensor(t, n, q_rot.shape)
    _check_tensor(lse, "lse", (B, L, H), torch.float32)
    dq, dk, dv = torch.empty_like(q_rot), torch.empty_like(q_rot), torch.empty_like(q_rot)
    if _empty(q_rot):
        return dq, dk, dv
    docs = _doclens(cu_doclens, B, L, q_rot.device)
    need = workspace_bytes(B, L, H, D)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q_rot.device)
    st = lib().dd_attn_bwd_rope(_ptr(q_rot), _ptr(k_rot), _ptr(v), _ptr(o), _ptr(do), _ptr(lse),
                                _ptr(dq), _ptr(dk), _ptr(dv), B, L, H, D, int(bool(causal)),
                                _ptr(docs.dev) if docs else None, docs.n_docs if docs else 0,
                                float(base), int(bool(doc_positions)), _ptr(workspace),
                                workspace.numel() * workspace.element_size(),
                                _stream(q_rot.device))
    check(st, "dd_attn_bwd_rope")
    return dq, dk, dv


class DDAttnFunction(torch.autograd.Function):
    """Autograd wrapper: forward saves (q, k, v, o, lse) for the backward, with
    q and k rotated when a RoPE base is given."""

    @staticmethod
    def forward(ctx, q, k, v, causal, cu_doclens, rope_base, rope_doc_positions):
        B, L = q.shape[0], q.shape[1]
        docs = _doclens(cu_doclens, B, L, q.device)
        if rope_base:
            o, lse, q, k = forward_rope(q, k, v, rope_base, causal, docs, rope_doc_positions)
        else:
            o, lse = forward(q, k, v, causal, docs)
        ctx.save_for_backward(q, k, v, o, lse)
        ctx.causal = causal
        ctx.docs = docs
        ctx.rope = (rope_base, rope_doc_positions)
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse = ctx.saved_tensors
        base, docpos = ctx.rope
        if base:
            dq, dk, dv = backward_rope(q, k, v, o, lse, do.contiguous(), base, ctx.causal,
                                       ctx.docs, docpos)
        else:
            dq, dk, dv = backward(q, k, v, o, lse, do.contiguous(), ctx.causal, ctx.docs)
        return dq, dk, dv, None, None, None, None


def attention(q, k, v, causal: bool = True, cu_doclens=None, rope_base=None,
              rope_doc_positions: bool = False):
    """Differentiable masked causal attention on [B, L, H, D] bf16 tensors;
    with ``rope_base`` the queries and keys are rotated first (RoPE)."""
    return DDAttnFunction.apply(q, k, v, causal, cu_doclens, rope_base, rope_doc_positions)
