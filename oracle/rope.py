"""fp64 oracle for rotary position embedding (RoPE) around the attention path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library and never imports it.

What it computes (arXiv 2405.13226, Sec. 3, paragraph "Positional
encoding"): queries and keys are rotated before attention.  Consecutive
components (2j, 2j+1) of a head vector form one pair, rotated by the angle
pos * f_b^(-2j/D) with base frequency f_b (10,000 in most runs, 100,000 in
the curriculum and scaling runs).  The rotation is the RoFormer definition the
paper cites:
    y_2j   = x_2j cos(a) - x_2j+1 sin(a)
    y_2j+1 = x_2j sin(a) + x_2j+1 cos(a),      a = pos * f_b^(-2j/D)
Attention then runs on the rotated q and k; the backward returns gradients
with respect to the unrotated q and k, i.e. the transposed rotation applied to
the gradients of the rotated ones.

Positions (the paper is silent; reading): a token's index within its row (the
DD sequence, or the concat-and-chunk chunk), or with ``doc_positions`` its
index from the start of its document inside the row, so that every DD piece
and every document of a masked chunk starts at position 0.
"""
from __future__ import annotations

import numpy as np

from . import attn_bwd as _attn_bwd
from . import attn_fwd as _attn_fwd


def widen(x) -> np.ndarray:
    """uint16 bf16 bit patterns -> float64 (exact); float input -> float64."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def positions(B: int, L: int, cu_doclens=None, doc_positions: bool = False) -> np.ndarray:
    """[B, L] int64 positions of every token (see module docstring)."""
    pos = np.tile(np.arange(L, dtype=np.int64), (B, 1))
    if not doc_positions or cu_doclens is None:
        return pos
    cu = [int(c) for c in cu_doclens]
    for b in range(B):
        for i in range(L):
            t = b * L + i
            start = max(c for c in cu[:-1] if c <= t)  # the document's first token
            pos[b, i] = t - max(start, b * L)          # clipped to the row
    return pos


def angles(pos, D: int, base: float) -> np.ndarray:
    """pos[...] -> [..., D/2] angles pos * base^(-2j/D) in float64."""
    j = np.arange(D // 2, dtype=np.float64)
    theta = np.power(float(base), -2.0 * j / D)
    return np.asarray(pos, dtype=np.float64)[..., None] * theta


def rotate(x, ang, inverse: bool = False) -> np.ndarray:
    """Rotate pairs (2j, 2j+1) of the last axis of x by ang[..., j]."""
    x = np.asarray(x, dtype=np.float64)
    c, s = np.cos(ang), np.sin(ang)
    if inverse:
        s = -s
    x0, x1 = x[..., 0::2], x[..., 1::2]
    y = np.empty_like(x)
    y[..., 0::2] = x0 * c - x1 * s
    y[..., 1::2] = x0 * s + x1 * c
    return y


def rope(x, base: float, cu_doclens=None, doc_positions: bool = False,
         inverse: bool = False) -> np.ndarray:
    """RoPE of a [B, L, H, D] tensor (bf16 bits or float), float64 result."""
    x = widen(x)
    B, L, H, D = x.shape
    ang = angles(positions(B, L, cu_doclens, doc_positions), D, base)  # [B, L, D/2]
    return rotate(x, ang[:, :, None, :], inverse)


def _pairs(bh, B, H):
    if bh is None:
        return [(b, h) for b in range(B) for h in range(H)]
    return [tuple(p) for p in bh]


def attn_fwd(q, k, v, base: float, causal: bool = True, cu_doclens=None,
             doc_positions: bool = False, bh=None):
    """Attention over rotated q and k.  Returns (o, lse), each [n_bh, L(, D)]."""
    qr = rope(q, base, cu_doclens, doc_positions)
    kr = rope(k, base, cu_doclens, doc_positions)
    return _attn_fwd(qr, kr, widen(v), causal, cu_doclens, bh)


def attn_bwd(q, k, v, do, base: float, causal: bool = True, cu_doclens=None,
             doc_positions: bool = False, bh=None):
    """Gradients of sum(dO * O) with respect to the unrotated q, k and v.

    Returns (dq, dk, dv), each [n_bh, L, D] in the order of ``bh``.
    """
    q, k = widen(q), widen(k)
    B, L, H, D = q.shape
    qr = rope(q, base, cu_doclens, doc_positions)
    kr = rope(k, base, cu_doclens, doc_positions)
    dqr, dkr, dv = _attn_bwd(qr, kr, widen(v), widen(do), causal, cu_doclens, bh)
    ang = angles(positions(B, L, cu_doclens, doc_positions), D, base)  # [B, L, D/2]
    dq = np.empty_like(dqr)
    dk = np.empty_like(dkr)
    for p, (b, _h) in enumerate(_pairs(bh, B, H)):
        dq[p] = rotate(dqr[p], ang[b], inverse=True)
        dk[p] = rotate(dkr[p], ang[b], inverse=True)
    return dq, dk, dv
