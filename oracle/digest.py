"""Content digests of a deposited artifact -- test infrastructure (see ``oracle/__init__``).

The paper verifies every graft by SHA-256 equality of bytes (Eq. 1) and identifies stored
blocks by their SHA-256 digests (Sec. 4.11); its deposit-side deduplication and hashing
machinery is closed (Sec. 3.1).  This module fixes the plain definitions the GPU digests must
reproduce bit for bit:

* ``leaf_digests``  the payload cut into consecutive leaves of ``leaf_bytes`` (the last one
                    may be shorter), each leaf's SHA-256 (FIPS 180-4) -- a content address
                    that any SHA-256 tool can recompute;
* ``merkle_root``   a binary tree over the leaf digests, level by level: nodes 2i and 2i+1
                    of a level combine into SHA-256(0x01 || left || right), a level's odd
                    last node moves up unchanged, the root of one leaf is its digest;
* ``dedup_map``     for every leaf, the smallest index of a leaf with the same digest.

SHA-256 itself is the standard library's (a library primitive used as a step), pinned by
the published FIPS 180 example digests in ``tests/golden/sha256_fips180_examples.txt``.
"""

from __future__ import annotations

import hashlib

import numpy as np

NODE_PREFIX = b"\x01"


def sha256(data: bytes) -> bytes:
    return hashlib.sha256(data).digest()


def leaf_digests(payload, leaf_bytes: int) -> np.ndarray:
    """[n_leaves][32] uint8 SHA-256 digests of consecutive ``leaf_bytes`` leaves."""
    buf = np.ascontiguousarray(payload).view(np.uint8).reshape(-1).tobytes()
    if leaf_bytes <= 0 or leaf_bytes % 64 or len(buf) == 0:
        raise ValueError("leaf_bytes must be a positive multiple of 64 and the payload non-empty")
    n = (len(buf) + leaf_bytes - 1) // leaf_bytes
    out = np.empty((n, 32), dtype=np.uint8)
    for i in range(n):
        out[i] = np.frombuffer(sha256(buf[i * leaf_bytes:(i + 1) * leaf_bytes]), dtype=np.uint8)
    return out


def merkle_root(digests) -> bytes:
    """Root of the level-by-level binary tree over 32-byte digests."""
    level = [bytes(d) for d in np.asarray(digests, dtype=np.uint8).reshape(-1, 32)]
    if not level:
        raise ValueError("no leaves")
    while len(level) > 1:
        nxt = [sha256(NODE_PREFIX + level[i] + level[i + 1]) for i in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


def dedup_map(digests) -> np.ndarray:
    """For each leaf, the smallest leaf index with an identical digest (int64)."""
    d = np.asarray(digests, dtype=np.uint8).reshape(-1, 32)
    first: dict[bytes, int] = {}
    out = np.empty(len(d), dtype=np.int64)
    for i, row in enumerate(d):
        out[i] = first.setdefault(row.tobytes(), i)
    return out
