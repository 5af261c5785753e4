"""The fresh computation of a workload, oracle side (test infrastructure only).

The paper's guarantee (Sec. 3.2, Eq. 1) compares the graft path against a fresh
computation of the same prefix: the block occupies [0, N) at its own
positions and the suffix and decode queries are computed on top.  With
synthetic K/V (no model weights) the "fresh" state of layer l is simply the
raw keys rotated at their absolute positions and rounded to the storage dtype,
plus the raw values; the outputs compared are the attention outputs of every
suffix row and every decode step.

Relocation (Sec. 4.2): a block captured at own_pos and grafted at target_pos
has its stored keys rotated by d = target_pos - own_pos.  ``relocated_kv``
gives those keys; ``fresh_kv`` at positions start_pos + t gives the fresh
reference at the new offset against which the residual is reported.
"""

from __future__ import annotations

import numpy as np

from synth.workloads import ROLE_K, ROLE_Q, ROLE_V, Workload, raw_rows

from .attention import attend
from .numerics import bits_to_values, round_to
from .rope import rotate, rotate_by


def fresh_kv(w: Workload, s: int, layers, n_keys: int, start_pos: int):
    """Cache contents of a fresh computation: K' = round(R(pos) k), V = round(v) (the
    rounding to the storage dtype is the identity for V unless the cache is fp8 and the
    raw values bf16), [L][n][Hkv][D] fp64."""
    k = bits_to_values(raw_rows(w, ROLE_K, s, layers, 0, n_keys), w.raw_dtype)
    v = bits_to_values(raw_rows(w, ROLE_V, s, layers, 0, n_keys), w.raw_dtype)
    pos = start_pos + np.arange(n_keys, dtype=np.float64)
    k_rot = round_to(rotate(k, pos, w.rope_base), w.dtype)
    return k_rot, round_to(v, w.dtype)


def relocated_kv(w: Workload, s: int, layers, n_block: int, n_keys: int):
    """Cache after a relocated graft: block keys captured at own_pos, rotated by
    d = start_pos - own_pos and rounded; tokens after the block computed fresh at
    start_pos + t."""
    k_own, v = fresh_kv(w, s, layers, n_keys, w.own_pos)
    d = w.start_pos - w.own_pos
    k_blk = round_to(rotate_by(k_own[:, :n_block], d, w.rope_base), w.dtype)
    k_new, _ = fresh_kv(w, s, layers, n_keys, w.start_pos)
    k_new[:, :n_block] = k_blk
    return k_new, v


def query_rows(w: Workload, s: int, layers, rows, start_pos: int):
    """Rotated queries for logical rows (fp64, [L][len(rows)][Hq][D])."""
    rows = np.asarray(rows, dtype=np.int64)
    out = []
    for (lo, hi) in _runs(rows):
        q = bits_to_values(raw_rows(w, ROLE_Q, s, layers, lo, hi - lo), w.raw_dtype)
        out.append(rotate(q, start_pos + np.arange(lo, hi, dtype=np.float64), w.rope_base))
    return np.concatenate(out, axis=1)


def _runs(rows):
    """Split a sorted row list into contiguous [lo, hi) runs."""
    runs = []
    start = prev = int(rows[0])
    for r in rows[1:]:
        r = int(r)
        if r != prev + 1:
            runs.append((start, prev + 1))
            start = r
        prev = r
    runs.append((start, prev + 1))
    return runs


def expected_rows(w: Workload, s: int, layers, rows, start_pos=None, kv=None):
    """Oracle attention outputs [L][len(rows)][Hq][D] for logical rows of sequence s.

    Each row i attends keys [0, i] of the fresh cache (suffix prefill and decode
    alike), or (i - W, i] in a layer with sliding window W.  ``kv`` may supply precomputed (K', V) covering max(rows) + 1 keys.
    """
    layers = list(layers)
    rows = np.asarray(sorted(rows), dtype=np.int64)
    sp = w.start_pos if start_pos is None else start_pos
    n_keys = int(rows.max()) + 1
    if kv is None:
        kv = fresh_kv(w, s, layers, n_keys, sp)
    k, v = kv
    q = query_rows(w, s, layers, rows, sp)
    return np.stack([attend(q[i], rows, k[i, :n_keys], v[i, :n_keys], w.scale, w.layer_window(layers[i]))
                     for i in range(len(layers))])
