"""Causal grouped-query softmax attention, oracle side (test infrastructure only).

After a graft the restored block is the prefix [0, N) of a fresh context and new
queries are computed on top of it (Sec. 3.2); the suffix prompt is prefilled in
a chunk and decoding advances one token at a time (Sec. 4.3).  Both are the
same operation for a query row at logical index i:

    s_j = (q_h . k_{g(h), j}) * scale      for every key j <= i  (inclusive causal)
    o_h = sum_j softmax(s)_j v_{g(h), j}

with q already rotated at its absolute position, keys stored rotated, and the
grouped-query head map g(h) = h // (Hq / Hkv) (contiguous groups).  fp64
throughout, softmax with the row maximum subtracted.  A decode step appends
its token's k/v first and then attends inclusively, so it is the row at the
new token's index.

The paper's model interleaves sliding-window layers with global ones and keeps a
full-size cache for the windowed layers (Sec. 4.3): a windowed layer with window
W > 0 restricts row i to the keys i - W < j <= i; W = 0 is full causal attention.
"""

from __future__ import annotations

import numpy as np


def attend(q: np.ndarray, q_index: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
           window: int = 0) -> np.ndarray:
    """q: [T][Hq][D] fp64 (rotated); q_index: [T] logical index of each row;
    k, v: [S][Hkv][D] fp64 in logical order (S > max(q_index)); window: 0 for full causal
    attention, W > 0 for keys (i - W, i].  Returns [T][Hq][D]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    T, Hq, D = q.shape
    S, Hkv, _ = k.shape
    group = Hq // Hkv
    q_index = np.asarray(q_index, dtype=np.int64)
    if q_index.max(initial=-1) >= S:
        raise ValueError("query row beyond the keys")
    if window < 0:
        raise ValueError("window must be >= 0")
    j = np.arange(S)[None, :]
    mask = j > q_index[:, None]                               # [T][S] True = not visible
    if window > 0:
        mask |= j <= q_index[:, None] - window
    out = np.empty((T, Hq, D), dtype=np.float64)
    for h in range(Hq):
        g = h // group
        s = (q[:, h, :] @ k[:, g, :].T) * scale              # [T][S]
        s = np.where(mask, -np.inf, s)
        m = s.max(axis=1, keepdims=True)
        p = np.exp(s - m)
        out[:, h, :] = (p @ v[:, g, :]) / p.sum(axis=1, keepdims=True)
    return out


def attend_paged(q, q_index, pool, block_table, n_keys, layer, scale, window: int = 0):
    """Same as ``attend`` with keys/values read from a paged pool through a block table."""
    from .numerics import bits_to_values
    k_bits, v_bits = pool.read_tokens(block_table, 0, n_keys)
    k = bits_to_values(k_bits[layer], pool.dtype)
    v = bits_to_values(v_bits[layer], pool.dtype)
    return attend(q, q_index, k, v, scale, window)
