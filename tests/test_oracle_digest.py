"""Pins of the digest oracle: the published FIPS 180 SHA-256 examples, an independent
recursive formulation of the tree for power-of-two leaf counts, the odd-node rule on small
trees, order sensitivity, and the dedup map against a brute-force comparison of raw leaf
bytes (not digests)."""

import os

import numpy as np
import pytest

from oracle import digest as od

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "sha256_fips180_examples.txt")


def _examples():
    out = []
    for ln in open(GOLDEN):
        ln = ln.split("#")[0].strip()
        if not ln:
            continue
        msg, hexd = ln.split()
        if msg == "<empty>":
            m = b""
        elif msg.startswith("a*"):
            m = b"a" * int(msg[2:])
        else:
            m = msg.encode()
        out.append((m, hexd))
    return out


@pytest.mark.parametrize("msg,hexd", _examples(), ids=lambda x: str(len(x)) if isinstance(x, bytes) else x[:8])
def test_sha256_fips_examples(msg, hexd):
    assert od.sha256(msg).hex() == hexd


def test_leaf_split_and_ragged_tail():
    rng = np.random.default_rng(1)
    buf = rng.integers(0, 256, size=5 * 128 + 64, dtype=np.uint8)      # 5 full leaves + 64 bytes
    d = od.leaf_digests(buf, 128)
    assert d.shape == (6, 32)
    assert d[5].tobytes() == od.sha256(buf[640:].tobytes())
    assert d[2].tobytes() == od.sha256(buf[256:384].tobytes())
    with pytest.raises(ValueError):
        od.leaf_digests(buf, 100)


def _recursive_root(ds):
    """Independent formulation for 2^k leaves: hash the two halves' roots."""
    if len(ds) == 1:
        return ds[0]
    h = len(ds) // 2
    return od.sha256(b"\x01" + _recursive_root(ds[:h]) + _recursive_root(ds[h:]))


@pytest.mark.parametrize("n", [1, 2, 4, 8, 64])
def test_merkle_power_of_two_matches_recursive(n):
    rng = np.random.default_rng(n)
    ds = [rng.integers(0, 256, size=32, dtype=np.uint8).tobytes() for _ in range(n)]
    assert od.merkle_root(np.frombuffer(b"".join(ds), np.uint8)) == _recursive_root(ds)


def test_merkle_odd_nodes_and_order():
    rng = np.random.default_rng(7)
    a, b, c = (rng.integers(0, 256, size=32, dtype=np.uint8).tobytes() for _ in range(3))
    arr = lambda *xs: np.frombuffer(b"".join(xs), np.uint8)  # noqa: E731
    # three leaves: the third moves up and pairs with the first pair's node
    ab = od.merkle_root(arr(a, b))
    assert od.merkle_root(arr(a, b, c)) == od.merkle_root(arr(ab, c))
    # five leaves: ((ab, cd), e)
    d, e = (rng.integers(0, 256, size=32, dtype=np.uint8).tobytes() for _ in range(2))
    cd = od.merkle_root(arr(c, d))
    assert od.merkle_root(arr(a, b, c, d, e)) == od.merkle_root(arr(od.merkle_root(arr(ab, cd)), e))
    assert od.merkle_root(arr(a, b)) != od.merkle_root(arr(b, a))
    assert od.merkle_root(arr(a)) == a


def test_dedup_map_against_raw_bytes():
    rng = np.random.default_rng(3)
    base = rng.integers(0, 256, size=(6, 256), dtype=np.uint8)
    order = [0, 1, 2, 1, 3, 0, 4, 5, 5, 2]                              # planted repeats
    buf = base[order].reshape(-1)
    got = od.dedup_map(od.leaf_digests(buf, 256))
    leaves = buf.reshape(len(order), 256)
    want = [min(j for j in range(len(order)) if np.array_equal(leaves[j], leaves[i])) for i in range(len(order))]
    assert got.tolist() == want
