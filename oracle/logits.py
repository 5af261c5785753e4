"""Logit head and the distribution statistics of the exactness test -- test infrastructure
(see ``oracle/__init__``).

The paper's verdict on a graft is taken on the logits at a position: byte equality of the
logit vectors (SHA-256, Eq. 1), and as corollaries a zero KL divergence between the two
softmax distributions and equal argmax (Eq. 2), reported over 50 samples together with a
Mann-Whitney U test against the noise floor and Cliff's delta (Sec. 4.1's table).  Its
model ends in a logit soft cap, through which small differences are amplified (Sec. 4.2).
This module fixes the plain definitions:

* ``logit_head``     a synthetic head over a hidden vector: the hidden value rounded to
                     bf16 (nearest, ties to even), z = W h exactly (fp64 here, W's bf16
                     values exact), logits = cap * tanh(z / cap), or z when cap = 0;
* ``kl_divergence``  KL(p || q) = sum_i p_i (log p_i - log q_i) with p = softmax(a),
                     q = softmax(b), in fp64 from the fp32 logits;
* ``argmax``         the first index of the largest logit;
* ``mann_whitney_u`` U of sample x against y: pairs with x_i > y_j count 1, ties 1/2;
* ``cliffs_delta``   (#(x_i > y_j) - #(x_i < y_j)) / (|x| |y|).

Pins (``tests/test_oracle_logits.py``): the tanh closed form tanh(ln(3) / 2) = 1/2, the
soft cap's limits, ties-to-even rounding of the hidden value, a hand-computed non-square
product, the two-point KL closed forms in both directions, shift invariance, first-index
ties, and the U statistic and its two-sided p-value against the textbook small-sample
values and scipy's implementation.
"""

from __future__ import annotations

import numpy as np

from .numerics import round_bf16


def logit_head(hidden: np.ndarray, w: np.ndarray, cap: float) -> np.ndarray:
    """hidden: [R][H] fp32 values; w: [V][H] weight values (on the bf16 grid); cap >= 0.
    Returns [R][V] fp64 logits."""
    h = round_bf16(np.asarray(hidden, dtype=np.float32).astype(np.float64))
    z = h @ np.asarray(w, dtype=np.float64).T
    if cap == 0:
        return z
    if cap < 0:
        raise ValueError("cap must be >= 0")
    return cap * np.tanh(z / cap)


def log_softmax(a: np.ndarray) -> np.ndarray:
    a = np.asarray(a, dtype=np.float64)
    m = a.max(axis=-1, keepdims=True)
    return a - m - np.log(np.exp(a - m).sum(axis=-1, keepdims=True))


def kl_divergence(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """KL(softmax(a) || softmax(b)) over the last axis (fp64)."""
    la, lb = log_softmax(a), log_softmax(b)
    return (np.exp(la) * (la - lb)).sum(axis=-1)


def argmax(a: np.ndarray) -> np.ndarray:
    """First index of the maximum over the last axis."""
    return np.argmax(np.asarray(a), axis=-1)


def mann_whitney_u(x, y) -> float:
    x = np.asarray(x, dtype=np.float64)[:, None]
    y = np.asarray(y, dtype=np.float64)[None, :]
    return float((x > y).sum() + 0.5 * (x == y).sum())


def mann_whitney_p(x, y) -> float:
    """Two-sided p-value of U under the normal approximation with the tie correction and
    a continuity correction of 1/2; 1.0 when every value is tied (no variance)."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    n1, n2 = len(x), len(y)
    n = n1 + n2
    u = mann_whitney_u(x, y)
    _, counts = np.unique(np.concatenate([x, y]), return_counts=True)
    var = n1 * n2 / 12.0 * ((n + 1) - (counts ** 3 - counts).sum() / (n * (n - 1)))
    if var <= 0:
        return 1.0
    mu = n1 * n2 / 2.0
    z = max(abs(u - mu) - 0.5, 0.0) / np.sqrt(var)
    from math import erfc, sqrt
    return min(1.0, erfc(z / sqrt(2.0)))


def cliffs_delta(x, y) -> float:
    x = np.asarray(x, dtype=np.float64)[:, None]
    y = np.asarray(y, dtype=np.float64)[None, :]
    return float(((x > y).sum() - (x < y).sum()) / (x.size * y.size))
