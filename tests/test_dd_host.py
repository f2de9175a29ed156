"""Host-side step shaping of the library against the oracle's independent
versions (binary decomposition, segments, useful pairs)."""
import numpy as np
import pytest

from oracle import decompose as odec
from oracle import metrics as omet
from paper_2405_13226_amd import dd
import synth


@pytest.mark.parametrize("length", [1, 2, 5, 255, 256, 257, 600, 4095, 8192, 8193, 20000])
@pytest.mark.parametrize("min_len,max_len", [(1, None), (256, 8192), (64, 1024)])
def test_binary_pieces_match_oracle(length, min_len, max_len):
    ours = dd.binary_pieces(length, min_len, max_len)
    ref = odec.pieces_of(length, min_len, max_len if max_len else 1 << 62)
    assert ours == ref


@pytest.mark.parametrize("seed", range(5))
def test_decompose_lognormal_documents(seed):
    lens = synth.lognormal_doc_lengths(seed)
    buckets = dd.decompose(lens, min_len=256, max_len=8192)
    ref = odec.decompose(lens, min_len=256, max_len=8192)
    assert sorted(buckets) == sorted(ref)
    starts = np.concatenate([[0], np.cumsum(lens)])
    for n, b in buckets.items():
        exp = [starts[d] + off for d, off, _ in ref[n]]
        np.testing.assert_array_equal(b.starts, exp)
    kept = sum(n * b.count for n, b in buckets.items())
    # Tokens kept are what remains after dropping pieces shorter than 256.
    assert kept == sum(sum(n for _, n in odec.pieces_of(int(x), 256, 8192)) for x in lens)
    assert 0.8 * 65536 < kept <= 65536


def test_every_token_in_exactly_one_piece():
    lens = synth.lognormal_doc_lengths(11, total_tokens=20000)
    cover = np.zeros(20000, dtype=np.int64)
    for n, b in dd.decompose(lens).items():
        for s in b.starts:
            cover[s:s + n] += 1
    assert np.all(cover == 1)


@pytest.mark.parametrize("seed", range(4))
def test_useful_pairs_match_oracle(seed):
    rng = np.random.default_rng(seed)
    B, L = int(rng.integers(1, 5)), int(rng.integers(1, 40))
    cu = np.unique(np.concatenate([[0, B * L], rng.integers(1, B * L, 5)]))
    for causal in (True, False):
        for c in (None, cu):
            assert dd.useful_pairs(B, L, causal, c) == omet.allowed_pairs_bruteforce(B, L, causal, c)


def test_chunk_doclens_and_vsl():
    lens = synth.lognormal_doc_lengths(0)
    cu = dd.chunk_doclens(lens, 65536)
    assert cu[0] == 0 and cu[-1] == 65536 and np.all(np.diff(cu) > 0)
    assert [dd.vsl_batch(65536, 2 ** i) for i in range(8, 14)] == [256, 128, 64, 32, 16, 8]
    with pytest.raises(ValueError):
        dd.vsl_batch(65536, 3000)


def test_flops_and_bytes():
    f, b = dd.attention_flops(8, 8192, 16, 128)
    pairs = 8 * 16 * 8192 * 8193 // 2
    assert f == 4 * 128 * pairs and b == 10 * 128 * pairs
    fb, bb = dd.attention_bytes(256, 256, 16, 64)
    t = 65536 * 16 * 64 * 2
    assert fb == 4 * t + 65536 * 16 * 4 and bb == 8 * t + 65536 * 16 * 4


@pytest.mark.parametrize("seed", range(3))
def test_packed_step_matches_buckets(seed):
    lens = synth.lognormal_doc_lengths(seed)
    packed = dd.pack_step(lens, min_len=256, max_len=8192)
    buckets = dd.decompose(lens, min_len=256, max_len=8192)
    assert packed.tokens == sum(n * b.count for n, b in buckets.items())
    # every packed piece is a contiguous run of source tokens of its bucket length
    cu = packed.cu_doclens
    assert cu[0] == 0 and cu[-1] == packed.tokens and np.all(np.diff(cu) >= 256)
    assert np.all(cu % 128 == 0)  # no kernel tile straddles two pieces
    for a, z in zip(cu[:-1], cu[1:]):
        run = packed.src[a:z]
        assert np.all(np.diff(run) == 1)
    # shortest pieces first
    assert np.all(np.diff(packed.lengths) >= 0)
    # the same multiset of pieces as the per-bucket decomposition
    got = sorted(zip(packed.src[cu[:-1]].tolist(), np.diff(cu).tolist()))
    ref = sorted((int(s), n) for n, b in buckets.items() for s in b.starts)
    assert got == ref
