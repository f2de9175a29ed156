"""Token-level decomposition and Algorithm 1 (length-based sampling and
curriculum), checked against the properties the paper states:
* every token appears in exactly one bucket, pieces are adjacent and their
  lengths are the binary digits of the document length (Sec. 2.1);
* every step holds b tokens of one bucket, b / 2^i sequences (Sec. 2.2);
* each cycle uses n_i / c tokens of bucket i, so the number of steps of
  bucket i per cycle is n_i / (c b) (Algorithm 1);
* sequences are drawn without replacement, subsets of different cycles do
  not overlap;
* the first draw of a cycle follows the odds (Table "curriculum").
"""
import numpy as np
import pytest

from paper_2405_13226_amd import sampler
import synth


def make_docs(seed, n_docs=400):
    rng = np.random.default_rng(seed)
    lens = synth.lognormal_doc_lengths(seed, total_tokens=600_000, median=900)[:n_docs]
    docs, nxt = [], 0
    for ell in lens:
        docs.append(np.arange(nxt, nxt + int(ell), dtype=np.int64))  # unique token ids
        nxt += int(ell)
    return docs, rng


def test_every_token_in_exactly_one_bucket():
    docs, _ = make_docs(0)
    tb = sampler.TokenBuckets.from_documents(docs)
    seen = np.concatenate([a.ravel() for a in tb.seqs.values()])
    total = sum(d.size for d in docs)
    assert seen.size == total
    assert np.array_equal(np.sort(seen), np.arange(total))
    for L, a in tb.seqs.items():
        assert L & (L - 1) == 0 and a.shape[1] == L
        assert np.all(np.diff(a, axis=1) == 1)  # a piece is a contiguous run of one document


@pytest.mark.parametrize("name,cycles", [("grow_p2", 8), ("uniform", 1), ("grow_linear", 2)])
def test_algorithm_1_steps(name, cycles):
    docs, rng = make_docs(1, n_docs=2000)
    tb = sampler.TokenBuckets.from_documents(docs, min_len=256, max_len=8192)
    b = 8192
    lengths = [L for L in sampler.CURRICULUM_LENGTHS if tb.tokens(L) >= cycles * b]
    n = {L: (tb.tokens(L) // (cycles * b)) * cycles * b for L in lengths}
    odds = {L: sampler.preset_odds(name)[L] for L in lengths}
    steps = list(sampler.curriculum_steps(tb.rows(), n, odds, cycles, b, rng))
    assert len(lengths) >= 3
    used = {L: [] for L in lengths}
    for st in steps:
        assert st.rows.size * st.length == b  # b tokens per step, b / 2^i sequences
        used[st.length].append(st.rows)
    for L in lengths:
        rows = np.concatenate(used[L]) if used[L] else np.zeros(0, int)
        assert rows.size * L == n[L]  # n_i tokens over all cycles
        assert np.unique(rows).size == rows.size  # without replacement
        per_cycle = [sum(s.rows.size for s in steps if s.length == L and s.cycle == j)
                     for j in range(cycles)]
        assert all(p * L == n[L] // cycles for p in per_cycle)  # n_i / (c b) steps per cycle
    # cycles are consecutive in the step order
    cyc = [s.cycle for s in steps]
    assert cyc == sorted(cyc)


def test_first_draw_follows_odds():
    docs, _ = make_docs(2, n_docs=3000)
    tb = sampler.TokenBuckets.from_documents(docs, min_len=256, max_len=8192)
    b = 2048
    lengths = [256, 512, 1024]
    n = {L: b * 2 for L in lengths}
    odds = {256: 4, 512: 2, 1024: 1}
    first = []
    for s in range(3000):
        rng = np.random.default_rng(s)
        st = next(sampler.curriculum_steps(tb.rows(), n, odds, 1, b, rng))
        first.append(st.length)
    frac = np.array([np.mean(np.array(first) == L) for L in lengths])
    assert np.allclose(frac, [4 / 7, 2 / 7, 1 / 7], atol=0.03)


def test_rejects_impossible_requests():
    docs, rng = make_docs(3, n_docs=50)
    tb = sampler.TokenBuckets.from_documents(docs, min_len=256, max_len=8192)
    with pytest.raises(ValueError):
        list(sampler.curriculum_steps(tb.rows(), {256: 10 ** 9}, {256: 1}, 1, 1024, rng))
    with pytest.raises(ValueError):
        list(sampler.curriculum_steps(tb.rows(), {512: 1024}, {512: 1}, 1, 1000, rng))
