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


# ---------------------------------------------------------------- fp8 E4M3 (OCP FP8 spec)
from oracle.numerics import fp8_bits_to_values, fp8_values_to_bits, round_fp8  # noqa: E402


def test_fp8_published_constants():
    # OCP 8-bit floating point specification, E4M3: bias 7, max 448 = 0x7E, min normal 2^-6
    # = 0x08, min subnormal 2^-9 = 0x01, 1.0 = 0x38, NaN = 0x7F / 0xFF, no infinities
    v = fp8_bits_to_values(np.array([0x38, 0x7E, 0x08, 0x01, 0x07, 0x80, 0xFE, 0x00], dtype=np.uint8))
    assert list(v) == [1.0, 448.0, 2.0 ** -6, 2.0 ** -9, 7 * 2.0 ** -9, -0.0, -448.0, 0.0]
    assert np.signbit(v[5])
    assert np.isnan(fp8_bits_to_values(np.array([0x7F, 0xFF], dtype=np.uint8))).all()
    codes = np.arange(256, dtype=np.uint8)
    vals = fp8_bits_to_values(codes)
    fin = ~np.isnan(vals)
    assert fin.sum() == 254
    pos = vals[:0x7F]                                   # 0x00 .. 0x7E ascend strictly
    assert np.all(np.diff(pos) > 0)
    assert np.array_equal(fp8_values_to_bits(vals[fin]), codes[fin])
    assert np.array_equal(round_fp8(vals[fin]), vals[fin])


def test_fp8_ties_to_even_and_saturation():
    # grid step 1/8 in [1, 2): 1 + 1/16 is a tie -> 1 (even mantissa), 1 + 3/16 -> 1.25
    assert round_fp8(np.array([1 + 1 / 16, 1 + 3 / 16, 1 + 1 / 16 + 1e-9])).tolist() == [1.0, 1.25, 1.125]
    # subnormal ties: 2^-10 -> 0 (even), 3 * 2^-10 -> 2 * 2^-9 (even), just above 2^-10 -> 2^-9
    assert round_fp8(np.array([2.0 ** -10, 3 * 2.0 ** -10, 2.0 ** -10 + 1e-12])).tolist() == [0.0, 2.0 ** -8, 2.0 ** -9]
    # the largest normal binade [256, 448]: step 32; 432 is a tie between 416 and 448 -> 448
    assert round_fp8(np.array([432.0, 400.0, 460.0, 1e6, -1e6])).tolist() == [448.0, 384.0, 448.0, 448.0, -448.0]
    assert np.signbit(round_fp8(np.array([-1e-5])))[0]


def test_fp8_matches_torch_in_range():
    import torch
    rng = np.random.default_rng(8)
    x = np.concatenate([rng.normal(size=50_000) * 40, rng.normal(size=50_000) * 0.01,
                        rng.uniform(-448, 448, size=20_000)]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    ours = fp8_values_to_bits(round_fp8(x.astype(np.float64)))
    assert np.array_equal(ref, ours)


def test_f32_ties_to_even_literals():
    # fp32 has 24 significant bits: in [1, 2) the grid step is 2^-23, so 1 + 2^-24 is a tie
    # between 1 (even) and 1 + 2^-23 (odd) and rounds down; 1 + 3 * 2^-24 lies between
    # 1 + 2^-23 (odd) and 1 + 2^-22 (even) and rounds up; a value just above a tie rounds up
    # (a truncating or ties-away cast fails one of these)
    x = np.array([1 + 2**-24, 1 + 3 * 2**-24, 1 + 2**-24 + 2**-40, 1 + 2**-24 - 2**-40,
                  -(1 + 3 * 2**-24), 2**100 * (1 + 2**-24), 2**-30 * (1 + 3 * 2**-24),
                  1.5 * (1 + 2**-24)])
    # the last value: 1.5 + 1.5 * 2^-24 is three quarters of a step above 1.5 and rounds up
    want = [1.0, 1 + 2**-22, 1 + 2**-23, 1.0, -(1 + 2**-22), 2.0**100, 2**-30 * (1 + 2**-22), 1.5 + 2**-23]
    assert round_f32(x).tolist() == want
    # values already on the grid are unchanged, and the result is always on the grid
    r = round_f32(np.random.default_rng(6).standard_normal(1000) * 1e3)
    assert np.array_equal(r.astype(np.float32).astype(np.float64), r)
