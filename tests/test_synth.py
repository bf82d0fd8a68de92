"""The seeded input generators: determinism, bf16 rounding, distributions."""

import numpy as np

from paper_2606_18114_amd import synth


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 0.0, -0.0, 3.0e38], np.float32)
    bits = synth.f32_to_bf16_bits(x)
    # 1+2^-8 is the tie between 1.0 (even) and 1+2^-7; 1+3*2^-8 ties up to 1+2^-6
    assert bits.tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x0000, 0x8000, 0x7F62]
    np.testing.assert_array_equal(synth.bf16_bits_to_f32(bits[:4]),
                                  np.array([1.0, 1.0, 1 + 2 ** -6, -2.5], np.float32))


def test_generators_are_deterministic():
    a = synth.single_linear_inputs(synth.C1)
    b = synth.single_linear_inputs(synth.C1)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    assert a[0].shape == (256, 512) and a[1].shape == (16, 512)


def test_weight_distribution_with_outliers():
    W = synth.weights(np.random.default_rng(0), 512, 2048, outliers=True)
    big = np.abs(W) > 0.2          # ~10 sigma of the bulk: essentially all outliers
    frac = np.mean(np.abs(W) > 0.12)
    assert 0.002 < big.mean() < 0.01 and 0.005 < frac < 0.015
    core = W[np.abs(W) < 0.1]
    assert abs(core.std() - 0.02) < 0.002
