"""Pins for the oracle's storage rounding."""

import numpy as np
import pytest

from oracle.numerics import bits_to_values, round_bf16, round_f32, values_to_bits


def test_bf16_ties_to_even_literals():
    assert round_bf16(np.array([1 + 2**-8]))[0] == 1.0                  # tie -> even (down)
    assert round_bf16(np.array([1 + 3 * 2**-8]))[0] == 1 + 2**-6        # tie -> even (up)
    assert round_bf16(np.array([-(1 + 2**-8)]))[0] == -1.0
    assert round_bf16(np.array([0.0]))[0] == 0.0
    assert round_bf16(np.array([255.5]))[0] == 256.0


def test_bf16_direct_rounding_no_double_rounding():
    # just above a bf16 tie but below fp32 resolution: must round up; going through
    # fp32 first would land exactly on the tie and round down.
    x = np.array([1 + 2**-8 + 2**-40])
    assert round_bf16(x)[0] == 1 + 2**-7


def test_bf16_matches_torch_on_fp32_inputs():
    torch = pytest.importorskip("torch")
    x = (np.random.default_rng(3).standard_normal(50_000) * 3).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(round_bf16(x.astype(np.float64)), ref)


def test_f32_and_bits_round_trip():
    x = np.random.default_rng(4).standard_normal(1000)
    r = round_f32(x)
    assert np.array_equal(bits_to_values(values_to_bits(r, "f32"), "f32"), r)
    b = round_bf16(x)
    assert np.array_equal(bits_to_values(values_to_bits(b, "bf16"), "bf16"), b)
    with pytest.raises(ValueError):
        values_to_bits(np.array([1 + 2**-12]), "bf16")
