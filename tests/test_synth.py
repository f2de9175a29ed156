"""The seeded input generators: bf16 rounding and workload shapes."""
import numpy as np
import pytest
import torch

import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10 ** rng.uniform(-6, 6, 100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 65504.0, 3.4e38, -3.4e38, 1e-40],
                                 dtype=np.float32)])
    ours = synth.bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = synth.f32_from_bf16_bits(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(ours.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_ties_round_to_even():
    # 1 + 2^-8 is exactly halfway between bf16 1.0 and 1.0078125: goes to 1.0
    assert synth.bf16_bits_from_f32(np.float32([1.00390625]))[0] == 0x3F80
    # 1 + 3*2^-8 is halfway between 1.0078125 (odd) and 1.015625 (even)
    assert synth.bf16_bits_from_f32(np.float32([1.01171875]))[0] == 0x3F82


def test_inputs_are_seeded_and_distinct():
    a = synth.attention_inputs(2, 8, 2, 4, seed=3)
    b = synth.attention_inputs(2, 8, 2, 4, seed=3)
    for n in a:
        np.testing.assert_array_equal(a[n], b[n])
    assert not np.array_equal(a["q"], a["k"])
    big = synth.f32_from_bf16_bits(synth.normal_bf16((200000,), 0, 1))
    assert abs(big.mean()) < 0.01 and abs(big.std() - 1) < 0.01


@pytest.mark.parametrize("seed", range(5))
def test_lognormal_documents_fill_the_step(seed):
    lens = synth.lognormal_doc_lengths(seed)
    assert lens.sum() == 65536
    assert lens.min() >= 1 and lens.max() <= 8192
    assert 40 < len(lens) < 120


def test_length_stream_weights():
    s = synth.length_stream(0)
    assert len(s) == 64
    vals, counts = np.unique(s, return_counts=True)
    assert set(vals) <= {256, 512, 1024, 2048, 4096, 8192, 16384}
    many = synth.length_stream(1, steps=200000)
    frac = (many == 256).mean()
    w = 1 / np.array([256, 512, 1024, 2048, 4096, 8192, 16384])
    assert abs(frac - w[0] / w.sum()) < 0.01
