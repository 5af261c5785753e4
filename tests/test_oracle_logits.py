"""Pins of the oracle's logit head and distribution statistics (Sec. 3.2 Eq. 1-2, Sec. 4.1's
table, the soft cap of Sec. 4.2) against closed forms, hand-computed values and scipy."""

import math

import numpy as np
import pytest
import scipy.stats

from oracle.logits import (argmax, cliffs_delta, kl_divergence, logit_head, mann_whitney_p,
                           mann_whitney_u)


def test_softcap_closed_form():
    # tanh(ln(3) / 2) = (3 - 1) / (3 + 1) = 1/2: with z = 1 and cap = 2 / ln 3 the logit is cap / 2
    cap = 2.0 / math.log(3.0)
    got = logit_head(np.array([[1.0]], np.float32), np.array([[1.0]]), cap)
    assert got[0, 0] == pytest.approx(cap / 2, rel=1e-15)


def test_softcap_limits():
    w = np.eye(3)
    h = np.array([[0.0, 8192.0, -8192.0]], np.float32)
    got = logit_head(h, w, 30.0)[0]
    assert got[0] == 0.0
    assert got[1] == pytest.approx(30.0, rel=1e-15) and got[2] == pytest.approx(-30.0, rel=1e-15)
    # small z: cap tanh(z / cap) = z - z^3 / (3 cap^2) + ...
    z = 2.0 ** -6
    got = logit_head(np.array([[z]], np.float32), np.array([[1.0]]), 30.0)[0, 0]
    assert got == pytest.approx(z - z ** 3 / (3 * 900.0), rel=1e-12)
    assert got < z
    # cap 0: the raw product (of the hidden value on the bf16 grid: 10000 -> 9984)
    assert logit_head(np.array([[1e4]], np.float32), np.array([[1.0]]), 0.0)[0, 0] == 9984.0


def test_hidden_rounds_to_bf16_ties_to_even():
    # bf16 spacing at 1 is 2^-7: 1 + 2^-8 is a tie (-> 1), 1 + 3 * 2^-8 a tie (-> 1 + 2^-6),
    # 1 + 2^-8 + 2^-20 rounds up, and -(1 + 2^-8) keeps its sign
    h = np.array([[1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -(1 + 2 ** -8)]], np.float32)
    got = logit_head(h, np.eye(4), 0.0)[0]
    assert list(got) == [1.0, 1 + 2 ** -6, 1 + 2 ** -7, -1.0]


def test_nonsquare_product_by_hand():
    w = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, -6.0]])
    h = np.array([[1.0, 2.0], [0.5, -1.0]], np.float32)
    assert logit_head(h, w, 0.0).tolist() == [[5.0, 11.0, -7.0], [-1.5, -2.5, 8.5]]


def test_kl_two_point_closed_forms():
    a = np.array([0.0, 0.0])                 # p = (1/2, 1/2)
    b = np.array([0.0, math.log(3.0)])       # q = (1/4, 3/4)
    assert kl_divergence(a, b) == pytest.approx(0.5 * math.log(4.0 / 3.0), rel=1e-14)
    assert kl_divergence(b, a) == pytest.approx(0.25 * math.log(0.5) + 0.75 * math.log(1.5), rel=1e-14)


def test_kl_identity_shift_and_sign():
    rng = np.random.default_rng(3)
    a = rng.normal(size=(6, 1000)) * 5
    b = a + rng.normal(size=a.shape) * 0.1
    assert np.all(kl_divergence(a, a) == 0.0)
    assert np.allclose(kl_divergence(a + 7.0, b - 2.0), kl_divergence(a, b), rtol=1e-10, atol=1e-15)
    assert np.all(kl_divergence(a, b) > 0)


def test_argmax_first_of_ties():
    assert argmax(np.array([1.0, 3.0, 3.0, -1.0])) == 1
    assert list(argmax(np.array([[0.0, 0.0], [2.0, 5.0]]))) == [0, 1]


def test_mann_whitney_textbook_and_scipy():
    x, y = [1, 2, 3, 4, 5], [6, 7, 8, 9, 10]
    assert mann_whitney_u(x, y) == 0.0 and mann_whitney_u(y, x) == 25.0
    assert cliffs_delta(x, y) == -1.0 and cliffs_delta(y, x) == 1.0
    # identical samples (the graft's zero KLs against a zero noise floor): p = 1, delta = 0
    z = np.zeros(50)
    assert mann_whitney_u(z, z) == 1250.0 and mann_whitney_p(z, z) == 1.0 and cliffs_delta(z, z) == 0.0
    rng = np.random.default_rng(0)
    a, b = np.round(rng.normal(size=30), 1), np.round(rng.normal(size=25) + 0.3, 1)   # with ties
    for u, v in ((x, y), (a, b)):
        ref = scipy.stats.mannwhitneyu(u, v, alternative="two-sided", method="asymptotic", use_continuity=True)
        assert mann_whitney_u(u, v) == ref.statistic
        assert mann_whitney_p(u, v) == pytest.approx(ref.pvalue, rel=1e-12)
