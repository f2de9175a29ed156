"""Pins of the oracle's length statistics, pair counts and decomposition.

* Table "mixture" (Sec. 3.3) prints, for seven DD mixtures, the tokens per
  bucket and the resulting average sequence and context lengths (Appendix F,
  eq. avg_context); the fixture tests/golden/mixture_table.txt holds them.
* Allowed-pair counts are checked by brute force over every (query, key).
* The binary decomposition (Sec. 2.1) is checked against its defining
  properties: every token in exactly one piece, piece lengths are the binary
  digits of the document length, pieces adjacent.
"""
import os

import numpy as np
import pytest

from oracle import decompose, metrics

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mixture_table.txt")


def load_mixture():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            parts = line.split()
            tokens = [int(x) for x in parts[1:9]]
            rows.append((parts[0], tokens, int(parts[9]), int(parts[10])))
    return rows


@pytest.mark.parametrize("name,tokens,seq,ctx", load_mixture())
def test_mixture_table_averages(name, tokens, seq, ctx):
    per_bucket = {2 ** (6 + i): t for i, t in enumerate(tokens) if t}
    got_seq, got_ctx = metrics.bucket_stats(per_bucket)
    assert abs(got_seq - seq) <= 0.5, (name, got_seq)
    assert abs(got_ctx - ctx) <= 0.5, (name, got_ctx)


def test_avg_ctx_literal_matches_bucket_form():
    lens = [64] * 3 + [1024] * 2 + [8192]
    a = metrics.avg_ctx_len(lens)
    b = metrics.bucket_stats({64: 3 * 64, 1024: 2 * 1024, 8192: 8192})[1]
    assert abs(a - b) < 1e-9
    assert metrics.avg_seq_len(lens) == pytest.approx(sum(lens) / len(lens))


@pytest.mark.parametrize("seed", range(6))
def test_allowed_pairs_match_brute_force(seed):
    rng = np.random.default_rng(seed)
    B, L = int(rng.integers(1, 4)), int(rng.integers(1, 30))
    cuts = np.unique(np.concatenate([[0, B * L], rng.integers(0, B * L, 4)]))
    for causal in (True, False):
        for cu in (None, cuts):
            assert metrics.allowed_pairs(B, L, causal, cu) == \
                metrics.allowed_pairs_bruteforce(B, L, causal, cu)
    # causal pairs = (avg ctx + 1) * tokens (Appendix F)
    segs = metrics.row_segments(B, L, cuts)
    pairs = metrics.allowed_pairs(B, L, True, cuts)
    assert pairs == pytest.approx((metrics.avg_ctx_len(segs) + 1) * B * L)


@pytest.mark.parametrize("length", [1, 2, 3, 255, 256, 600, 1023, 4097, 8191, 8192, 12345])
def test_binary_pieces(length):
    pieces = decompose.pieces_of(length)
    lens = [n for _, n in pieces]
    assert sum(lens) == length
    assert len(pieces) == bin(length).count("1")
    assert all(n & (n - 1) == 0 for n in lens)
    assert sorted(lens, reverse=True) == lens
    off = 0
    for o, n in pieces:
        assert o == off
        off += n


def test_pieces_min_and_max():
    p = decompose.pieces_of(8192 + 8192 + 300, min_len=256, max_len=8192)
    assert p == [(0, 8192), (8192, 8192), (16384, 256)]
    b = decompose.decompose([300, 1000, 255], min_len=256)
    assert sorted(b) == [256, 512]
    assert [x[0] for x in b[256]] == [0, 1]
