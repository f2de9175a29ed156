"""Token-level dataset decomposition and the length-based sampler/curriculum.

* ``TokenBuckets.from_documents`` -- Sec. 2.1: every tokenized document is cut
  into the adjacent pieces of its binary decomposition; piece lengths 2^i go
  to bucket D_i, so every token lands in exactly one bucket.
* ``curriculum_steps`` -- Algorithm 1 (Appendix B.2): training runs in ``c``
  cycles; each cycle uses a fresh, disjoint random subset of every bucket
  holding n_i / c of its tokens, and each of its steps takes b / 2^i unused
  sequences of one bucket, the bucket chosen with probability proportional
  to its odds o_i among the buckets the cycle has not used up.  Every step
  therefore holds b tokens of one sequence length (Sec. 2.2, VSL).
* ``ODDS`` -- the sampling odds of Table "curriculum" for D_8..D_13.

Readings where the paper is silent: a cycle's subset of bucket i holds
floor(n_i / (c * b)) whole steps (so every step has exactly b tokens; tokens
beyond that are not used), subsets are drawn uniformly without replacement,
and sequences within a subset are consumed in a uniformly shuffled order.
Random draws come from a numpy Generator passed by the caller.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .dd import binary_pieces

# Sampling odds for buckets D_8 .. D_13 (sequence lengths 256 .. 8192).
ODDS = {
    "uniform": (1, 1, 1, 1, 1, 1),
    "grow_linear": (6, 5, 4, 3, 2, 1),
    "grow_p2": (32, 16, 8, 4, 2, 1),
    "grow_p100": (100 ** 5, 100 ** 4, 100 ** 3, 100 ** 2, 100, 1),
    "shrink_p100": (1, 100, 100 ** 2, 100 ** 3, 100 ** 4, 100 ** 5),
}
CURRICULUM_LENGTHS = (256, 512, 1024, 2048, 4096, 8192)


@dataclass
class TokenBuckets:
    """Bucket length -> [n_seq, length] array of token ids (one row per piece)."""

    seqs: dict = field(default_factory=dict)

    @staticmethod
    def from_documents(docs, min_len: int = 1, max_len: int | None = None) -> "TokenBuckets":
        rows: dict = {}
        for d in docs:
            d = np.asarray(d)
            for off, n in binary_pieces(d.size, min_len, max_len):
                rows.setdefault(n, []).append(d[off:off + n])
        return TokenBuckets({n: np.stack(r) for n, r in sorted(rows.items())})

    def tokens(self, length: int) -> int:
        a = self.seqs.get(length)
        return 0 if a is None else int(a.size)

    def rows(self) -> dict:
        """Bucket length -> number of sequences."""
        return {n: int(a.shape[0]) for n, a in self.seqs.items()}


@dataclass
class Step:
    cycle: int
    length: int
    rows: np.ndarray  # indices into TokenBuckets.seqs[length]


def _bucket_order(steps: dict, odds: dict, rng: np.random.Generator) -> list:
    """Bucket length of every step of one cycle.

    The sampling rule: each step goes to a bucket that still has steps left
    in the cycle, chosen with probability proportional to its odds among
    those buckets; a cycle ends when every bucket's steps are used.
    """
    left = {L: n for L, n in steps.items() if n > 0}
    order = []
    while left:
        live = sorted(left)
        w = np.array([float(odds[L]) for L in live])
        L = live[int(rng.choice(len(live), p=w / w.sum()))]
        order.append(L)
        left[L] -= 1
        if left[L] == 0:
            del left[L]
    return order


def curriculum_steps(rows_per_bucket: dict, tokens_per_bucket: dict, odds: dict,
                     cycles: int, tokens_per_step: int, rng: np.random.Generator):
    """Yield the steps of Algorithm 1 in training order.

    rows_per_bucket: number of sequences in the bucket of length L (key L),
    e.g. TokenBuckets.rows().  tokens_per_bucket: n_i, tokens to use from the
    bucket of length L.  odds: o_i per bucket length.  cycles: c.
    tokens_per_step: b.  Each step's ``rows`` index that bucket's sequences.
    """
    lengths = sorted(tokens_per_bucket)
    for L in lengths:
        if tokens_per_step % L:
            raise ValueError(f"b = {tokens_per_step} is not a multiple of {L}")
        need = tokens_per_bucket[L]
        have = rows_per_bucket.get(L, 0) * L
        if need > have:
            raise ValueError(f"bucket {L} holds {have} tokens, {need} requested")
    # A step of bucket L holds b / L sequences; a cycle uses n_L / c tokens of
    # it, i.e. n_L / (c b) whole steps.
    seqs_per_step = {L: tokens_per_step // L for L in lengths}
    steps = {L: tokens_per_bucket[L] // (cycles * tokens_per_step) for L in lengths}
    # The cycles' subsets of each bucket: disjoint, drawn uniformly at random
    # (one permutation of the bucket cut into consecutive runs), each holding
    # the sequences of that cycle's steps in the order they are consumed.
    subsets = {}
    for L in lengths:
        perm = rng.permutation(rows_per_bucket.get(L, 0))
        size = steps[L] * seqs_per_step[L]
        subsets[L] = [perm[j * size:(j + 1) * size] for j in range(cycles)]
    for j in range(cycles):
        used = {L: 0 for L in lengths}
        for L in _bucket_order(steps, odds, rng):
            k = used[L]
            used[L] += 1
            rows = subsets[L][j][k * seqs_per_step[L]:(k + 1) * seqs_per_step[L]]
            yield Step(cycle=j, length=L, rows=rows)


def preset_odds(name: str, lengths=CURRICULUM_LENGTHS) -> dict:
    return dict(zip(lengths, ODDS[name]))
