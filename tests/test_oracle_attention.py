"""Pins for the oracle's causal GQA attention: brute force and closed forms."""

import math

import numpy as np
import pytest

from oracle.attention import attend

rng = np.random.default_rng(17)


def brute_force(q, q_index, k, v, scale):
    """Element loops, softmax written as exp(s)/sum exp(s) with no max shift."""
    T, Hq, D = q.shape
    S, Hkv, _ = k.shape
    out = np.zeros((T, Hq, D))
    for t in range(T):
        for h in range(Hq):
            g = h * Hkv // Hq
            w = []
            for j in range(int(q_index[t]) + 1):
                s = 0.0
                for d in range(D):
                    s += float(q[t, h, d]) * float(k[j, g, d])
                w.append(math.exp(s * scale))
            z = sum(w)
            for d in range(D):
                out[t, h, d] = sum(w[j] * float(v[j, g, d]) for j in range(len(w))) / z
    return out


@pytest.mark.parametrize("Hq,Hkv", [(4, 2), (4, 4), (8, 2), (3, 1)])
def test_matches_brute_force(Hq, Hkv):
    D, S, T = 8, 9, 4
    q = rng.standard_normal((T, Hq, D))
    k = rng.standard_normal((S, Hkv, D))
    v = rng.standard_normal((S, Hkv, D))
    idx = np.array([0, 3, 5, 8])
    np.testing.assert_allclose(attend(q, idx, k, v, 0.3), brute_force(q, idx, k, v, 0.3), rtol=1e-12,
                               atol=1e-13)


def test_zero_query_gives_prefix_mean():
    S, D = 12, 16
    k = rng.standard_normal((S, 2, D))
    v = rng.standard_normal((S, 2, D))
    q = np.zeros((S, 4, D))
    o = attend(q, np.arange(S), k, v, 1.0)
    for i in range(S):
        np.testing.assert_allclose(o[i, 0], v[: i + 1, 0].mean(axis=0), rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(o[i, 3], v[: i + 1, 1].mean(axis=0), rtol=1e-13, atol=1e-14)


def test_first_row_sees_only_itself():
    # inclusive causality: row 0 has one visible key, so its output is v_0
    k = rng.standard_normal((5, 1, 8))
    v = rng.standard_normal((5, 1, 8))
    q = rng.standard_normal((1, 2, 8)) * 10
    o = attend(q, np.array([0]), k, v, 1.0)
    np.testing.assert_allclose(o[0, 0], v[0, 0], rtol=1e-14)
    np.testing.assert_allclose(o[0, 1], v[0, 0], rtol=1e-14)


def test_identical_keys_give_mean():
    k = np.tile(rng.standard_normal((1, 1, 8)), (6, 1, 1))
    v = rng.standard_normal((6, 1, 8))
    q = rng.standard_normal((1, 1, 8))
    o = attend(q, np.array([5]), k, v, 0.7)
    np.testing.assert_allclose(o[0, 0], v[:, 0].mean(axis=0), rtol=1e-13)


def test_needle_dominates():
    S, D = 50, 32
    k = rng.standard_normal((S, 1, D)) * 0.1
    v = rng.standard_normal((S, 1, D))
    q = rng.standard_normal((1, 1, D))
    k[17, 0] = q[0, 0] * 40.0                     # margin >> log(S)
    o = attend(q, np.array([S - 1]), k, v, 1.0)
    np.testing.assert_allclose(o[0, 0], v[17, 0], rtol=1e-8, atol=1e-8)


def test_future_keys_ignored():
    k = rng.standard_normal((10, 2, 8))
    v = rng.standard_normal((10, 2, 8))
    q = rng.standard_normal((2, 4, 8))
    idx = np.array([3, 6])
    o1 = attend(q, idx, k, v, 0.5)
    k2, v2 = k.copy(), v.copy()
    k2[7:] = 99.0
    v2[7:] = -99.0
    assert np.array_equal(attend(q, idx, k2, v2, 0.5), o1)


def test_gqa_contiguous_group_map():
    k = rng.standard_normal((6, 2, 8))
    v = rng.standard_normal((6, 2, 8))
    q = rng.standard_normal((1, 4, 8))
    o = attend(q, np.array([5]), k, v, 0.5)
    k2, v2 = k.copy(), v.copy()
    k2[:, 1] += 1.0
    v2[:, 1] += 1.0
    o2 = attend(q, np.array([5]), k2, v2, 0.5)
    assert np.array_equal(o[0, :2], o2[0, :2])        # heads 0, 1 read kv head 0
    assert not np.allclose(o[0, 2:], o2[0, 2:])       # heads 2, 3 read kv head 1
    # and each head equals single-head attention with its own kv head
    for h in range(4):
        single = attend(q[:, h:h + 1], np.array([5]), k[:, h // 2:h // 2 + 1], v[:, h // 2:h // 2 + 1], 0.5)
        np.testing.assert_allclose(o[0, h], single[0, 0], rtol=1e-14)


def test_shift_invariance():
    # adding the same vector c to every key adds q.c to every score of a row
    k = rng.standard_normal((7, 1, 8))
    v = rng.standard_normal((7, 1, 8))
    q = rng.standard_normal((3, 1, 8))
    c = rng.standard_normal(8) * 3
    idx = np.array([2, 4, 6])
    np.testing.assert_allclose(attend(q, idx, k + c, v, 0.8), attend(q, idx, k, v, 0.8), rtol=1e-12,
                               atol=1e-13)


def test_large_scores_stable():
    k = rng.standard_normal((5, 1, 4)) * 100
    v = rng.standard_normal((5, 1, 4))
    q = rng.standard_normal((1, 1, 4)) * 100
    assert np.all(np.isfinite(attend(q, np.array([4]), k, v, 1.0)))


def _brute_window(q, qi, k, v, scale, window):
    """Element loops, un-shifted softmax, for a sliding window."""
    T, Hq, D = q.shape
    group = Hq // k.shape[1]
    out = np.zeros_like(q)
    for t in range(T):
        for h in range(Hq):
            js = [j for j in range(qi[t] + 1) if window == 0 or j > qi[t] - window]
            ws = [np.exp(float(np.dot(q[t, h], k[j, h // group])) * scale) for j in js]
            tot = sum(ws)
            for wgt, j in zip(ws, js):
                out[t, h] += wgt / tot * v[j, h // group]
    return out


@pytest.mark.parametrize("window", [1, 3, 7, 20])
def test_sliding_window_brute_force(window):
    rng = np.random.default_rng(window)
    S, T = 20, 6
    q = rng.normal(size=(T, 4, 8))
    k, v = rng.normal(size=(S, 2, 8)), rng.normal(size=(S, 2, 8))
    qi = np.array([0, 2, 5, 9, 14, 19])
    got = attend(q, qi, k, v, 0.35, window)
    assert np.abs(got - _brute_window(q, qi, k, v, 0.35, window)).max() < 1e-12


def test_sliding_window_limits():
    rng = np.random.default_rng(9)
    S = 30
    q = rng.normal(size=(5, 2, 4))
    k, v = rng.normal(size=(S, 1, 4)), rng.normal(size=(S, 1, 4))
    qi = np.array([0, 7, 12, 28, 29])
    # a window covering every visible key is full causal attention
    assert np.array_equal(attend(q, qi, k, v, 0.5, 30), attend(q, qi, k, v, 0.5, 0))
    # window 1: each row sees only its own key
    got = attend(q, qi, k, v, 0.5, 1)
    assert np.allclose(got[:, 0], v[qi, 0], atol=1e-15)
    # keys before the window have no influence
    k2, v2 = k.copy(), v.copy()
    k2[:10] += 100.0
    v2[:10] = 1.0e6                                     # finite garbage: weight 0 times it is 0
    assert np.array_equal(attend(q[3:], qi[3:], k2, v2, 0.5, 15), attend(q[3:], qi[3:], k, v, 0.5, 15))


def test_workload_layer_windows():
    from synth.workloads import BLOCK12B, scaled
    w = scaled(BLOCK12B, sliding_window=1024, global_every=6)
    win = w.layer_windows
    assert len(win) == 48 and win[5] == 0 and win[11] == 0 and win[0] == 1024 and win.count(0) == 8
    assert scaled(BLOCK12B).layer_windows == (0,) * 48
