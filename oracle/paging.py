"""Paged KV pool, deposit and graft, oracle side (test infrastructure only).

Sec. 3.1-3.2 describe the graft engine at the behaviour level: a processed
prefix's KV state S is captured (deposit) as a persistent block and later
installed into a fresh context (graft) as a prefix at its own positions
[0, N), new queries being computed on top at [N, N + q).  The storage layout of
a block is closed; the layout below is this implementation's.

Pool: per layer, for K and for V, ``[n_pages][n_kv_heads][page_size][head_dim]``
of storage bits.  Token t of a sequence lives in physical page
``block_table[t // page_size]`` at row ``t % page_size``.

Payload of a block of n tokens starting at logical token ``first`` (a multiple
of page_size): ``[n_layers][2 (K, V)][ceil(n / page_size)][n_kv_heads][page_size][head_dim]``,
logical page order, rows at or beyond n in the last page set to zero.
"""

from __future__ import annotations

import numpy as np

from .numerics import bits_to_values, round_to, storage_np_dtype, values_to_bits
from .rope import rotate, rotate_by


class PagedPool:
    def __init__(self, n_layers, n_pages, n_kv_heads, page_size, head_dim, dtype, fill_bits=0):
        self.shape = (n_layers, n_pages, n_kv_heads, page_size, head_dim)
        self.page_size = page_size
        self.dtype = dtype
        nd = storage_np_dtype(dtype)
        self.k = np.full(self.shape, fill_bits, dtype=nd)
        self.v = np.full(self.shape, fill_bits, dtype=nd)

    def write_tokens(self, block_table, t0, k_bits, v_bits):
        """Store rows for logical tokens [t0, t0 + T); k_bits/v_bits: [L][T][Hkv][D]."""
        P = self.page_size
        for i in range(k_bits.shape[1]):
            t = t0 + i
            page = block_table[t // P]
            self.k[:, page, :, t % P, :] = k_bits[:, i]
            self.v[:, page, :, t % P, :] = v_bits[:, i]

    def read_tokens(self, block_table, t0, n):
        """Logical-order copy of tokens [t0, t0 + n): two arrays [L][n][Hkv][D] of bits."""
        P = self.page_size
        idx_page = np.array([block_table[t // P] for t in range(t0, t0 + n)], dtype=np.int64)
        idx_row = np.array([t % P for t in range(t0, t0 + n)], dtype=np.int64)
        k = self.k[:, idx_page, :, idx_row, :]  # advanced indexing -> [n][L][Hkv][D]
        v = self.v[:, idx_page, :, idx_row, :]
        return np.moveaxis(k, 0, 1), np.moveaxis(v, 0, 1)


def append_kv(pool: PagedPool, block_table, t0, k_raw_bits, v_raw_bits, pos, base, pairing="half",
              raw_dtype=None):
    """Fresh computation of K/V for new tokens: rotate k at its absolute position
    (fp64), round to the storage dtype, store k and v through the block table.

    k_raw_bits, v_raw_bits: [L][T][Hkv][D] bits of raw_dtype (default: the storage dtype;
    an fp8 pool takes bf16 inputs, and its values are rounded to fp8 too);
    pos: [T] absolute positions.
    """
    raw_dtype = pool.dtype if raw_dtype is None else raw_dtype
    k = bits_to_values(k_raw_bits, raw_dtype)
    k_rot = round_to(rotate(k, pos, base, pairing), pool.dtype)
    if raw_dtype == pool.dtype:
        v_bits = np.asarray(v_raw_bits)
    else:
        v_bits = values_to_bits(round_to(bits_to_values(v_raw_bits, raw_dtype), pool.dtype), pool.dtype)
    pool.write_tokens(block_table, t0, values_to_bits(k_rot, pool.dtype), v_bits)


def payload_pages(n_tokens: int, page_size: int) -> int:
    return -(-n_tokens // page_size)


def deposit(pool: PagedPool, block_table, first_token, n_tokens) -> np.ndarray:
    """State capture: gather the block's pages into one contiguous payload."""
    L, _, Hkv, P, D = pool.shape
    if first_token % P:
        raise ValueError("first_token must be page aligned")
    npg = payload_pages(n_tokens, P)
    out = np.zeros((L, 2, npg, Hkv, P, D), dtype=pool.k.dtype)
    for p in range(npg):
        src = block_table[first_token // P + p]
        rows = min(P, n_tokens - p * P)
        out[:, 0, p, :, :rows, :] = pool.k[:, src, :, :rows, :]
        out[:, 1, p, :, :rows, :] = pool.v[:, src, :, :rows, :]
    return out


def graft(pool: PagedPool, payload: np.ndarray, block_table, first_token, n_tokens):
    """State restore at own position: scatter the payload's rows into the pages
    named by the target block table (a byte move, so the result is exact)."""
    P = pool.page_size
    if first_token % P:
        raise ValueError("first_token must be page aligned")
    for p in range(payload.shape[2]):
        dst = block_table[first_token // P + p]
        rows = min(P, n_tokens - p * P)
        pool.k[:, dst, :, :rows, :] = payload[:, 0, p, :, :rows, :]
        pool.v[:, dst, :, :rows, :] = payload[:, 1, p, :, :rows, :]


def relocate_payload(payload: np.ndarray, n_tokens: int, d: int, base, dtype, pairing="half"):
    """Relocated graft (Sec. 4.2): the block's keys, stored after rotation at their
    own positions, are rotated by the offset d = target_pos - own_pos (fp64) and
    rounded to the storage dtype; values are unchanged.  Tail rows stay zero."""
    out = payload.copy()
    L, _, npg, Hkv, P, D = payload.shape
    k = bits_to_values(payload[:, 0], dtype)                      # [L][npg][Hkv][P][D]
    k_tok = np.moveaxis(k, 3, 2).reshape(L, npg * P, Hkv, D)      # [L][tokens][Hkv][D]
    k_new = round_to(rotate_by(k_tok, d, base, pairing), dtype)
    k_new[:, n_tokens:] = 0.0
    k_new = np.moveaxis(k_new.reshape(L, npg, P, Hkv, D), 2, 3)
    out[:, 0] = values_to_bits(k_new, dtype)
    return out
