"""numpy side of the seeded input generator (see the package docstring).

Philox4x32-10 as defined by Salmon et al. (SC'11): ten rounds of
  (c0, c1, c2, c3) -> (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0))
with the key bumped by the Weyl constants (W0, W1) between rounds.
"""

from __future__ import annotations

import dataclasses

import numpy as np

PHILOX_M0 = np.uint64(0xD2511F53)
PHILOX_M1 = np.uint64(0xCD9E8D57)
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85

_MASK32 = np.uint64(0xFFFFFFFF)

# Tensor roles: part of the Philox stream id.
ROLE_Q = 1
ROLE_K = 2
ROLE_V = 3
ROLE_W = 4      # weights of the synthetic logit head: "token" = vocabulary row, dim = hidden
ROLE_H = 5      # standalone hidden vectors for the logit head: "token" = row, dim = hidden
ROLE_NK = 6     # needle key row of a store block ("token" 0 of its own stream)
ROLE_NV = 7     # needle value row (the code a probe retrieves) of a store block

# Logical token stride per layer in the element index, so that the raw value of
# (layer, token, head, dim) does not depend on how a sequence is chunked into calls.
TOKEN_STRIDE = 1 << 26


def philox4x32_10(ctr: np.ndarray, key: tuple[int, int]) -> np.ndarray:
    """Philox4x32-10 block function.  ctr: (N, 4) uint32; returns (N, 4) uint32."""
    c = [np.asarray(ctr[:, i], dtype=np.uint64) for i in range(4)]
    k0 = int(key[0]) & 0xFFFFFFFF
    k1 = int(key[1]) & 0xFFFFFFFF
    for rnd in range(10):
        p0 = PHILOX_M0 * c[0]
        p1 = PHILOX_M1 * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        c = [hi1 ^ c[1] ^ np.uint64(k0), lo1, hi0 ^ c[3] ^ np.uint64(k1), lo0]
        if rnd != 9:
            k0 = (k0 + PHILOX_W0) & 0xFFFFFFFF
            k1 = (k1 + PHILOX_W1) & 0xFFFFFFFF
    return np.stack(c, axis=1).astype(np.uint32)


def irwin_hall12(words: np.ndarray) -> np.ndarray:
    """(N, 4) uint32 Philox words -> int32 z = sum of twelve 10-bit uniforms - 6138."""
    w = words.astype(np.int64)
    s = np.zeros(w.shape[0], dtype=np.int64)
    for j in range(4):
        for sh in (0, 10, 20):
            s += (w[:, j] >> sh) & 1023
    return (s - 6138).astype(np.int32)


@dataclasses.dataclass(frozen=True)
class Stream:
    """Identifies one raw tensor family: (workload id, role, unit).

    ``unit`` is a sequence id for per-sequence inputs or a store block id for
    store blocks.
    """

    workload: int
    role: int
    unit: int

    @property
    def id(self) -> int:
        return (self.workload << 48) | (self.role << 40) | self.unit


def normal_f32(seed: int, stream: int, index: np.ndarray, sigma_log2: int) -> np.ndarray:
    """fp32 values z * 2**(sigma_log2 - 10) for element indices ``index`` (uint64)."""
    index = np.asarray(index, dtype=np.uint64).reshape(-1)
    ctr = np.empty((index.size, 4), dtype=np.uint32)
    ctr[:, 0] = (index & _MASK32).astype(np.uint32)
    ctr[:, 1] = (index >> np.uint64(32)).astype(np.uint32)
    ctr[:, 2] = np.uint32(stream & 0xFFFFFFFF)
    ctr[:, 3] = np.uint32((stream >> 32) & 0xFFFFFFFF)
    z = irwin_hall12(philox4x32_10(ctr, (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)))
    return np.ldexp(z.astype(np.float32), sigma_log2 - 10).astype(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); inputs are finite."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))
    return (b >> np.uint64(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_tensor(seed: int, stream: Stream, layers, t0: int, n_tokens: int, n_heads: int,
                  head_dim: int, sigma_log2: int, dtype: str) -> np.ndarray:
    """Raw tensor [len(layers)][n_tokens][n_heads][head_dim] of one stream.

    Element (l, t, h, d) has index ((l * TOKEN_STRIDE + t) * n_heads + h) * head_dim + d,
    with t the logical token index in its sequence or block.  Returns storage
    bits: uint16 for "bf16", uint32 for "f32".
    """
    layers = np.asarray(list(layers), dtype=np.uint64)
    t = np.arange(t0, t0 + n_tokens, dtype=np.uint64)
    h = np.arange(n_heads, dtype=np.uint64)
    d = np.arange(head_dim, dtype=np.uint64)
    idx = (((layers[:, None, None, None] * np.uint64(TOKEN_STRIDE) + t[None, :, None, None])
            * np.uint64(n_heads) + h[None, None, :, None]) * np.uint64(head_dim)
           + d[None, None, None, :])
    vals = normal_f32(seed, stream.id, idx.reshape(-1), sigma_log2)
    shape = (len(layers), n_tokens, n_heads, head_dim)
    if dtype == "bf16":
        return f32_to_bf16_bits(vals).reshape(shape)
    if dtype == "f32":
        return vals.view(np.uint32).reshape(shape)
    raise ValueError(f"unknown dtype {dtype!r}")
