"""Binary dataset decomposition, oracle side (Sec. 2.1 of arXiv 2405.13226).

TEST INFRASTRUCTURE ONLY (see the package docstring).

A document of length l = 2^{i_1} + ... + 2^{i_k} (its binary expansion) is cut
into k adjacent pieces of lengths 2^{i_1}, ..., 2^{i_k}; piece j goes to bucket
D_{i_j}.  The paper does not fix the piece order; this reading takes the
largest piece first.  Pieces shorter than ``min_len`` are dropped (the
benchmark keeps buckets 2^8..2^13) and a document longer than ``max_len`` is
first cut into ``max_len`` pieces.
"""
from __future__ import annotations


def pieces_of(length: int, min_len: int = 1, max_len: int = 1 << 62) -> list:
    """[(offset within the document, piece length)] for one document."""
    out = []
    off = 0
    rest = int(length)
    while rest >= max_len:
        out.append((off, max_len))
        off += max_len
        rest -= max_len
    bit = 1
    while bit * 2 <= rest:
        bit *= 2
    while bit >= 1:
        if rest & bit:
            if bit >= min_len:
                out.append((off, bit))
            off += bit
        bit //= 2
    return out


def decompose(doc_lengths, min_len: int = 1, max_len: int = 1 << 62) -> dict:
    """Bucket -> list of (document index, offset, length) for all documents."""
    buckets: dict = {}
    for d, ell in enumerate(doc_lengths):
        for off, n in pieces_of(int(ell), min_len, max_len):
            buckets.setdefault(n, []).append((d, off, n))
    return buckets
