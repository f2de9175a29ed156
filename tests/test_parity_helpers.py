"""The GPU parity checks' own error measures, on the CPU.

A local error -- one wrong block of rows, or one wrong (b, h) slice -- must
fail the blockwise and per-slice bounds even where the pooled relative L2
error of the whole tensor stays under the tolerance.
"""
import numpy as np

from parity import BWD_RTOL, ROW_BLOCK, local_errors, rel_l2


def test_one_wrong_key_block_fails_blockwise_bound():
    rng = np.random.default_rng(5)
    ref = rng.standard_normal((3, 8192, 64))
    got = ref + 1e-4 * rng.standard_normal(ref.shape)
    got[1, 4096:4096 + ROW_BLOCK] *= 1.05  # one 128-row block 5% off
    assert rel_l2(got, ref) <= BWD_RTOL            # hidden in the pooled norm
    sl, bl, _ = local_errors(got, ref)
    assert sl <= BWD_RTOL < bl                     # caught by the block bound


def test_one_wrong_slice_fails_slice_bound():
    rng = np.random.default_rng(6)
    ref = rng.standard_normal((16, 256, 64))
    got = ref.copy()
    got[9] *= 1.035  # one slice of 16 is 3.5% off
    assert rel_l2(got, ref) <= BWD_RTOL
    sl, bl, _ = local_errors(got, ref)
    assert sl > BWD_RTOL and bl > BWD_RTOL


def test_zero_reference_blocks_use_absolute_error():
    ref = np.zeros((2, 300, 8))
    ref[0, :128] = 1.0
    got = ref.copy()
    got[1, 200, 3] = 3e-6
    sl, bl, za = local_errors(got, ref)
    assert sl == 0.0 and bl == 0.0 and za == 3e-6


def test_ragged_tail_joins_previous_block():
    rng = np.random.default_rng(7)
    ref = rng.standard_normal((1, 300, 8))
    got = ref.copy()
    got[0, 290:] += 0.5  # inside the 44-row tail, checked with rows 128..299
    _, bl, _ = local_errors(got, ref)
    assert bl > BWD_RTOL
    # a one-row tail (L = 129) is checked as part of a 129-row block
    ref = rng.standard_normal((1, 129, 8))
    got = ref.copy()
    got[0, 128] *= 1.03
    _, bl, _ = local_errors(got, ref)
    assert 0 < bl < BWD_RTOL
