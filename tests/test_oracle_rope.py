"""Pins for the oracle's rotary embedding and relocation (Sec. 4.2, RoFormer)."""

import os

import numpy as np
import pytest

from oracle.numerics import round_bf16
from oracle.rope import inv_freq, rotate, rotate_by

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(5)


def _closed_forms():
    out = []
    with open(os.path.join(GOLDEN, "rope_d4_closed_form.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            p = line.split()
            out.append((p[0], float(p[1]), [float(x) for x in p[2:]]))
    return out


@pytest.mark.parametrize("pairing,pos,expected", _closed_forms())
def test_literal_closed_form(pairing, pos, expected):
    x = np.array([1.0, 2.0, 3.0, 4.0]).reshape(1, 1, 4)
    y = rotate(x, np.array([pos]), 10000.0, pairing).reshape(-1)
    np.testing.assert_allclose(y, expected, rtol=1e-13, atol=1e-13)


def test_inv_freq_literal():
    # theta_i = base^(-2i/D): D = 8, base = 10000 -> 1, 0.1, 0.01, 0.001
    np.testing.assert_allclose(inv_freq(8, 10000.0), [1.0, 0.1, 0.01, 0.001], rtol=1e-15)


def test_pos_zero_is_identity():
    x = rng.standard_normal((3, 5, 2, 64))
    assert np.array_equal(rotate(x, np.zeros(5), 10000.0), x)
    assert np.array_equal(rotate(x, np.zeros(5), 10000.0, "interleaved"), x)


@pytest.mark.parametrize("pairing", ["half", "interleaved"])
def test_pair_norms_preserved(pairing):
    D = 64
    x = rng.standard_normal((1, 7, 3, D))
    pos = rng.integers(0, 3_000_000, 7)
    y = rotate(x, pos, 10000.0, pairing)
    if pairing == "half":
        nx = x[..., :D // 2] ** 2 + x[..., D // 2:] ** 2
        ny = y[..., :D // 2] ** 2 + y[..., D // 2:] ** 2
    else:
        nx = x[..., 0::2] ** 2 + x[..., 1::2] ** 2
        ny = y[..., 0::2] ** 2 + y[..., 1::2] ** 2
    np.testing.assert_allclose(ny, nx, rtol=1e-14)


def test_composition_and_inverse():
    x = rng.standard_normal((1, 4, 2, 128))
    a, b = 1234, 8192
    ab = rotate(rotate(x, np.full(4, a), 1e4), np.full(4, b), 1e4)
    np.testing.assert_allclose(ab, rotate(x, np.full(4, a + b), 1e4), atol=1e-12)
    back = rotate_by(rotate_by(x, 8192, 1e4), -8192, 1e4)
    np.testing.assert_allclose(back, x, atol=1e-12)


def test_relative_position_identity():
    # <R(m) q, R(n) k> = <R(m - n) q, k>: the exact-arithmetic fact behind Sec. 4.2
    q = rng.standard_normal((1, 1, 1, 256))
    k = rng.standard_normal((1, 1, 1, 256))
    for m, n in [(10, 3), (40_000, 8_192), (2_854_000, 2_850_000)]:
        lhs = np.sum(rotate(q, [m], 1e4) * rotate(k, [n], 1e4))
        rhs = np.sum(rotate(q, [m - n], 1e4) * k)
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(rhs)) * 100


def test_concat_invariant_bit_equal():
    x = rng.standard_normal((2, 40, 2, 64))
    full = rotate(x, np.arange(40), 1e4)
    parts = np.concatenate([rotate(x[:, :25], np.arange(25), 1e4),
                            rotate(x[:, 25:], np.arange(25, 40), 1e4)], axis=1)
    assert np.array_equal(full, parts)


def test_interleaved_is_permuted_half():
    D = 16
    x = rng.standard_normal((1, 3, 1, D))
    perm = np.concatenate([np.arange(0, D, 2), np.arange(1, D, 2)])   # interleaved -> half order
    y_int = rotate(x, np.array([3, 70, 900]), 1e4, "interleaved")
    y_half = rotate(x[..., perm], np.array([3, 70, 900]), 1e4, "half")
    assert np.array_equal(y_int[..., perm], y_half)


def test_relocated_bf16_within_one_ulp_of_fresh():
    # k captured at own position p and moved by d, vs fresh at p + d: equal in exact
    # arithmetic; after the extra rounding about a third of the bf16 keys differ, each by
    # at most a couple of ulps of its pair's norm.
    k = round_bf16(rng.standard_normal((1, 64, 4, 128)) * 0.5)
    pos = np.arange(64)
    stored = round_bf16(rotate(k, pos, 1e4))
    moved = round_bf16(rotate_by(stored, 8192, 1e4))
    fresh = round_bf16(rotate(k, pos + 8192, 1e4))
    # each rounding errs by at most half an ulp of the pair norm r (pairs i, i + D/2),
    # and rotation carries an error vector over with its norm unchanged
    r = np.sqrt(k[..., :64] ** 2 + k[..., 64:] ** 2)
    r = np.concatenate([r, r], axis=-1)
    ulp_r = np.ldexp(1.0, np.frexp(np.maximum(r, 1e-30))[1] - 8)
    assert np.all(np.abs(moved - fresh) <= 2.0 * ulp_r)
    assert np.any(moved != fresh)      # and it is genuinely not byte-exact (Sec. 4.2)
