"""Sequence-length statistics and useful-work counts (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Appendix F of arXiv 2405.13226 defines, for sequences of lengths l_1..l_N:
  * average sequence length  = (1/N) * sum_i l_i
  * average context length   = sum_i sum_{j=0}^{l_i-1} j / sum_i l_i
                             = sum_i l_i (l_i - 1) / (2 sum_i l_i)   (eq. avg_context)
A token at context position j attends to j + 1 keys (contexts 0..l-1 plus the
token itself), so the number of allowed causal (query, key) pairs of a segment
of length l is sum_{j=0}^{l-1} (j + 1), and over all segments it equals
(average context length + 1) * total tokens.
"""
from __future__ import annotations

import numpy as np


def avg_seq_len(lengths) -> float:
    """Mean length (1/N) sum l_i."""
    lens = np.asarray(lengths, dtype=np.float64)
    return float(lens.sum() / lens.size)


def avg_ctx_len(lengths) -> float:
    """Average context length, summed literally over context positions."""
    lens = np.asarray(lengths, dtype=np.int64)
    num = 0
    for ell in lens:
        num += int(ell) * (int(ell) - 1) // 2  # sum_{j=0}^{l-1} j, exact integer
    return float(num) / float(lens.sum())


def bucket_stats(tokens_per_bucket: dict) -> tuple:
    """(avg seq len, avg ctx len) of a DD mixture given tokens per bucket.

    ``tokens_per_bucket`` maps a sequence length 2^i to the number of tokens
    drawn from bucket D_i; the bucket holds tokens / 2^i sequences of length
    2^i.  Token counts may be fractional multiples of a unit (e.g. 2^30): the
    statistics are ratios and do not depend on the unit.
    """
    n_seq = 0.0
    tok = 0.0
    ctx_num = 0.0
    for ell, t in tokens_per_bucket.items():
        n = float(t) / float(ell)
        n_seq += n
        tok += float(t)
        ctx_num += n * ell * (ell - 1) / 2.0
    return tok / n_seq, ctx_num / tok


def allowed_pairs_bruteforce(B: int, L: int, causal: bool = True,
                             cu_doclens=None) -> int:
    """Count allowed (query, key) pairs per head by testing every pair."""
    total = 0
    for b in range(B):
        doc = np.zeros(L, dtype=np.int64)
        if cu_doclens is not None:
            cu = np.asarray(cu_doclens, dtype=np.int64)
            for i in range(L):
                t = b * L + i
                d = 0
                for kk in range(cu.size - 1):
                    if cu[kk] <= t:
                        d = kk
                doc[i] = d
        for i in range(L):
            for j in range(L):
                if causal and j > i:
                    continue
                if doc[i] == doc[j]:
                    total += 1
    return total


def row_segments(B: int, L: int, cu_doclens=None) -> list:
    """Lengths of the attention segments: documents cut at row boundaries."""
    segs = []
    for b in range(B):
        lo, hi = b * L, (b + 1) * L
        if cu_doclens is None:
            segs.append(L)
            continue
        cu = [int(x) for x in cu_doclens]
        for kk in range(len(cu) - 1):
            s, e = max(cu[kk], lo), min(cu[kk + 1], hi)
            if e > s:
                segs.append(e - s)
    return segs


def allowed_pairs(B: int, L: int, causal: bool = True, cu_doclens=None) -> int:
    """Allowed pairs per head from the segment lengths (any size)."""
    total = 0
    for ell in row_segments(B, L, cu_doclens):
        total += ell * (ell + 1) // 2 if causal else ell * ell
    return total
