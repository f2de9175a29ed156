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

Precision (the paper is silent; reading): the rotated q and k are bf16
tensors, as a bf16 training step materialises them, i.e. the exact rotation
rounded to the nearest bf16 (ties to even) before attention; with
``round_rotated=False`` they stay exact.  Everything else is float64.
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


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bf16 (8 significant bits, ties to
    even), returned as float64.  Finite, normal-range inputs."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m * 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.round(np.ldexp(m, 8)), e - 8)  # np.round: half to even


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
         inverse: bool = False, rows=None) -> np.ndarray:
    """RoPE of a [B, L, H, D] tensor (bf16 bits or float), float64 result.
    With ``rows`` (batch indices) only those rows are rotated; the others are
    left zero (for oracles that read only some rows)."""
    B, L, H, D = np.asarray(x).shape
    ang = angles(positions(B, L, cu_doclens, doc_positions), D, base)  # [B, L, D/2]
    if rows is None:
        return rotate(widen(x), ang[:, :, None, :], inverse)
    y = np.zeros((B, L, H, D), dtype=np.float64)
    for b in sorted(set(int(r) for r in rows)):
        y[b] = rotate(widen(np.asarray(x)[b]), ang[b][:, None, :], inverse)
    return y


def _pairs(bh, B, H):
    if bh is None:
        return [(b, h) for b in range(B) for h in range(H)]
    return [tuple(p) for p in bh]


def _rotated(x, base, cu_doclens, doc_positions, round_rotated, rows=None):
    y = rope(x, base, cu_doclens, doc_positions, rows=rows)
    return round_bf16(y) if round_rotated else y


def _rows(bh):
    return None if bh is None else [p[0] for p in bh]


def _widen_rows(x, rows):
    if rows is None:
        return widen(x)
    x = np.asarray(x)
    y = np.zeros(x.shape, dtype=np.float64)
    for b in sorted(set(rows)):
        y[b] = widen(x[b])
    return y


def attn_fwd(q, k, v, base: float, causal: bool = True, cu_doclens=None,
             doc_positions: bool = False, bh=None, round_rotated: bool = True):
    """Attention over rotated q and k.  Returns (o, lse), each [n_bh, L(, D)]."""
    rows = _rows(bh)
    qr = _rotated(q, base, cu_doclens, doc_positions, round_rotated, rows)
    kr = _rotated(k, base, cu_doclens, doc_positions, round_rotated, rows)
    return _attn_fwd(qr, kr, _widen_rows(v, rows), causal, cu_doclens, bh)


def attn_bwd(q, k, v, do, base: float, causal: bool = True, cu_doclens=None,
             doc_positions: bool = False, bh=None, round_rotated: bool = True):
    """Gradients of sum(dO * O) with respect to the unrotated q, k and v (the
    rounding of the rotated q, k counts as identity in the chain rule, as the
    straight-through cast of a bf16 training step does).

    Returns (dq, dk, dv), each [n_bh, L, D] in the order of ``bh``.
    """
    B, L, H, D = np.asarray(q).shape
    rows = _rows(bh)
    qr = _rotated(q, base, cu_doclens, doc_positions, round_rotated, rows)
    kr = _rotated(k, base, cu_doclens, doc_positions, round_rotated, rows)
    dqr, dkr, dv = _attn_bwd(qr, kr, _widen_rows(v, rows), _widen_rows(do, rows), causal,
                             cu_doclens, bh)
    ang = angles(positions(B, L, cu_doclens, doc_positions), D, base)  # [B, L, D/2]
    dq = np.empty_like(dqr)
    dk = np.empty_like(dkr)
    for p, (b, _h) in enumerate(_pairs(bh, B, H)):
        dq[p] = rotate(dqr[p], ang[b], inverse=True)
        dk[p] = rotate(dkr[p], ang[b], inverse=True)
    return dq, dk, dv
