"""Rotary position embedding, oracle side (test infrastructure only).

The paper's model encodes absolute position with rotary embeddings (RoFormer,
Su et al. 2021, cited in Sec. 4.2): each pair of components of a query or key
is rotated by pos * theta_i, theta_i = base**(-2i/D), i in [0, D/2).  Sec. 4.2
notes that attention then depends only on relative position in exact
arithmetic, and that relocating a captured block to another offset means
rotating its keys by the offset.

Pairing (the paper is silent): "half" pairs component i with i + D/2 (the
rotate-half form); "interleaved" pairs 2i with 2i + 1.  Everything here is
fp64: angle = pos * theta_i, cos and sin in fp64.
"""

from __future__ import annotations

import numpy as np


def inv_freq(head_dim: int, base: float) -> np.ndarray:
    """theta_i = base ** (-2 i / D), fp64, i in [0, D/2)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(np.float64(base), -2.0 * i / head_dim)


def _pair_index(head_dim: int, pairing: str):
    half = head_dim // 2
    if pairing == "half":
        a = np.arange(half)
        return a, a + half
    if pairing == "interleaved":
        a = np.arange(half) * 2
        return a, a + 1
    raise ValueError(pairing)


def rotate(x: np.ndarray, pos: np.ndarray, base: float, pairing: str = "half") -> np.ndarray:
    """Rotate x[..., T, H, D] (fp64) by angle pos[T] * theta_i on each pair.

    (a, b) -> (a cos(phi) - b sin(phi), a sin(phi) + b cos(phi)), phi = pos * theta_i.
    ``pos`` may be negative (used for relocation by a negative offset).
    """
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    ia, ib = _pair_index(D, pairing)
    phi = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq(D, base)[None, :]  # [T, D/2]
    c = np.cos(phi)[:, None, :]
    s = np.sin(phi)[:, None, :]
    a = x[..., ia]
    b = x[..., ib]
    out = np.empty_like(x)
    out[..., ia] = a * c - b * s
    out[..., ib] = a * s + b * c
    return out


def rotate_by(x: np.ndarray, d: int, base: float, pairing: str = "half") -> np.ndarray:
    """Rotate every row of x[..., T, H, D] by the same offset d (relocation, Sec. 4.2)."""
    T = x.shape[-3]
    return rotate(x, np.full(T, d, dtype=np.float64), base, pairing)
