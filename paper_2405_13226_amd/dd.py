"""Host-side step shaping for dataset decomposition (DD).

* ``binary_pieces`` / ``decompose``: Sec. 2.1 of arXiv 2405.13226 -- a
  document of length l = 2^{i_1} + ... + 2^{i_k} is cut into k adjacent
  pieces of those lengths, and the piece of length 2^i joins bucket D_i.  The
  order of the pieces inside a document is not fixed by the paper; here the
  largest comes first.  Pieces shorter than ``min_len`` are dropped and a
  document longer than ``max_len`` is first cut into ``max_len`` pieces.
* ``vsl_batch``: Sec. 2.2 -- a step drawn from bucket D_i holds b / 2^i
  sequences of length 2^i, so every step has b tokens.
* ``chunk_doclens``: the concat-and-chunk baseline (Sec. 1) -- documents are
  concatenated and cut into fixed-length rows; the document boundaries become
  the ``cu_doclens`` offsets of the document-masked attention.
* ``pack_step``: every DD piece of a step packed into one row with piece
  boundaries as ``cu_doclens``, so the whole DD step runs as a single
  document-masked launch instead of one launch per bucket.
* ``useful_pairs`` / ``attention_flops``: the work the masked attention must
  do.  A token at context position j (Appendix F) attends to j + 1 keys, so a
  causal segment of length l has l(l+1)/2 (query, key) pairs per head.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def binary_pieces(length: int, min_len: int = 1, max_len: int | None = None):
    """[(offset, piece length)] of one document, largest piece first."""
    length = int(length)
    out = []
    off = 0
    if max_len is not None:
        if max_len & (max_len - 1):
            raise ValueError("max_len must be a power of two")
        n_full, length = divmod(length, max_len)
        for _ in range(n_full):
            out.append((off, max_len))
            off += max_len
    for bit in range(max(length.bit_length() - 1, 0), -1, -1):
        n = 1 << bit
        if length & n:
            if n >= min_len:
                out.append((off, n))
            off += n
    return out


@dataclass
class Bucket:
    length: int        # sequence length 2^i of the bucket
    starts: np.ndarray  # start offset of every piece in the concatenated token stream

    @property
    def count(self) -> int:
        return int(self.starts.size)


def decompose(doc_lengths, min_len: int = 1, max_len: int | None = None) -> dict:
    """Bucket length -> Bucket of all pieces of the documents (concat order)."""
    starts: dict = {}
    doc_start = 0
    for ell in doc_lengths:
        for off, n in binary_pieces(int(ell), min_len, max_len):
            starts.setdefault(n, []).append(doc_start + off)
        doc_start += int(ell)
    return {n: Bucket(n, np.asarray(s, dtype=np.int64)) for n, s in sorted(starts.items())}


def vsl_batch(tokens_per_step: int, length: int) -> int:
    """Number of sequences of a VSL step of bucket ``length``."""
    if tokens_per_step % length:
        raise ValueError("the token budget must be a multiple of the sequence length")
    return tokens_per_step // length


def chunk_doclens(doc_lengths, total_tokens: int | None = None) -> np.ndarray:
    """cu_doclens (int32) of documents concatenated in order."""
    lens = np.asarray(doc_lengths, dtype=np.int64)
    cu = np.concatenate([[0], np.cumsum(lens)])
    if total_tokens is not None and cu[-1] != total_tokens:
        raise ValueError("documents do not fill the step exactly")
    return cu.astype(np.int32)


def segments(B: int, L: int, cu_doclens=None) -> np.ndarray:
    """Lengths of attention segments: documents cut at the row edges."""
    if cu_doclens is None:
        return np.full(B, L, dtype=np.int64)
    cu = np.asarray(cu_doclens, dtype=np.int64)
    edges = np.union1d(cu, np.arange(0, B * L + 1, L, dtype=np.int64))
    return np.diff(edges)


def useful_pairs(B: int, L: int, causal: bool = True, cu_doclens=None) -> int:
    """Allowed (query, key) pairs of one head."""
    seg = segments(B, L, cu_doclens)
    if causal:
        return int((seg * (seg + 1) // 2).sum())
    return int((seg * seg).sum())


def attention_flops(B: int, L: int, H: int, D: int, causal: bool = True,
                    cu_doclens=None) -> tuple:
    """(forward, backward) useful FLOPs: 4*D and 10*D per allowed pair and head."""
    pairs = useful_pairs(B, L, causal, cu_doclens) * H
    return 4 * D * pairs, 10 * D * pairs


def attention_bytes(B: int, L: int, H: int, D: int) -> tuple:
    """(forward, backward) algorithmic HBM bytes: each tensor touched once.

    Forward reads Q, K, V and writes O and LSE.  Backward reads Q, K, V, O,
    dO and LSE and writes dQ, dK and dV.
    """
    t = B * L * H * D * 2
    s = B * L * H * 4
    return 4 * t + s, 8 * t + s


@dataclass
class PackedStep:
    """All DD pieces of a step packed into one row, ready for one masked launch.

    ``src`` gives, for every packed token, its position in the concatenated
    document stream; ``cu_doclens`` marks the piece boundaries of the packed
    row.  Attention of the packed row under the document mask is exactly the
    per-bucket DD attention: pieces never attend to each other.  Pieces are
    ordered shortest first, so the heaviest query blocks (the ends of the
    longest pieces) come last, where the kernels' heaviest-first block order
    starts.  With every piece length a multiple of 128, no 128-query or 64-key
    tile of the kernels straddles two pieces.
    """

    src: np.ndarray
    cu_doclens: np.ndarray
    lengths: np.ndarray

    @property
    def tokens(self) -> int:
        return int(self.src.size)


def pack_step(doc_lengths, min_len: int = 256, max_len: int | None = 8192) -> PackedStep:
    """Pack the binary-decomposition pieces of ``doc_lengths`` into one row."""
    buckets = decompose(doc_lengths, min_len, max_len)
    starts, lens = [], []
    for n in sorted(buckets):
        for s in buckets[n].starts:
            starts.append(int(s))
            lens.append(int(n))
    lens_a = np.asarray(lens, dtype=np.int64)
    src = np.concatenate([np.arange(s, s + n, dtype=np.int64) for s, n in zip(starts, lens)]) \
        if lens else np.zeros(0, dtype=np.int64)
    cu = np.concatenate([[0], np.cumsum(lens_a)]).astype(np.int32)
    return PackedStep(src=src, cu_doclens=cu, lengths=lens_a)
