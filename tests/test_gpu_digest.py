"""Content digests on the GPU against the oracle: per-leaf SHA-256 bit for bit (the FIPS 180
examples, ragged last leaves, leaves of 64 B to 64 KiB), the Merkle root for odd and even
leaf counts, the dedup map on a payload with planted duplicate slabs, and the digests of a
deposited artifact against those of the pages it restores."""

import hashlib
import os

import numpy as np
import pytest
import torch

from oracle import digest as od

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "sha256_fips180_examples.txt")


@pytest.fixture(scope="module")
def kvg():
    from paper_2607_14431_amd import kvg
    return kvg


def _dev(buf: np.ndarray) -> torch.Tensor:
    t = torch.empty(max(len(buf), 16), dtype=torch.uint8, device="cuda")
    t[: len(buf)] = torch.from_numpy(np.ascontiguousarray(buf))
    return t


def _gpu_digests(kvg, buf: np.ndarray, leaf: int) -> np.ndarray:
    n = (len(buf) + leaf - 1) // leaf
    out = torch.empty((n, 32), dtype=torch.uint8, device="cuda")
    kvg.kvg_leaf_digests(_dev(buf), leaf, out, n_bytes=len(buf))
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_fips_examples(kvg):
    for ln in open(GOLDEN):
        ln = ln.split("#")[0].strip()
        if not ln:
            continue
        msg, hexd = ln.split()
        if msg == "<empty>":
            continue                                     # an empty buffer is rejected by the call
        m = b"a" * int(msg[2:]) if msg.startswith("a*") else msg.encode()
        leaf = (len(m) + 63) // 64 * 64                 # one leaf holding the whole message
        got = _gpu_digests(kvg, np.frombuffer(m, np.uint8), leaf)
        print(f"FIPS example of {len(m)} bytes", flush=True)
        assert got.shape == (1, 32) and got[0].tobytes().hex() == hexd


@pytest.mark.parametrize("n_bytes,leaf", [(5 * 4096 + 100, 4096), (64 * 333 + 55, 64), (64 * 333 + 56, 64),
                                          (8192 * 97, 8192), (65536 * 3 + 63, 65536), (12345, 12288)])
def test_leaf_digests_match_oracle(kvg, n_bytes, leaf):
    rng = np.random.default_rng(n_bytes)
    buf = rng.integers(0, 256, size=n_bytes, dtype=np.uint8)
    got = _gpu_digests(kvg, buf, leaf)
    want = od.leaf_digests(buf, leaf)
    print(f"{n_bytes} bytes in leaves of {leaf}: {len(want)} leaves", flush=True)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 64, 1000, 4097])
def test_merkle_root_matches_oracle(kvg, n):
    rng = np.random.default_rng(100 + n)
    d = rng.integers(0, 256, size=(n, 32), dtype=np.uint8)
    dev = torch.from_numpy(d).cuda()
    root = torch.zeros(32, dtype=torch.uint8, device="cuda")
    ws = torch.empty(kvg.kvg_merkle_workspace_bytes(n), dtype=torch.uint8, device="cuda")
    kvg.kvg_merkle_root(dev, n, root, ws)
    torch.cuda.synchronize()
    assert root.cpu().numpy().tobytes() == od.merkle_root(d)


def test_dedup_map_planted_duplicates(kvg):
    rng = np.random.default_rng(5)
    slab = 8192
    base = rng.integers(0, 256, size=(40, slab), dtype=np.uint8)
    order = rng.integers(0, 40, size=600)                       # ~560 repeats among 600 leaves
    buf = base[order].reshape(-1)
    dg = _gpu_digests(kvg, buf, slab)
    n = len(order)
    fi = torch.empty(n, dtype=torch.int64, device="cuda")
    unres = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    ws = torch.empty(kvg.kvg_dedup_workspace_bytes(n), dtype=torch.uint8, device="cuda")
    kvg.kvg_dedup_map(torch.from_numpy(dg).cuda(), n, fi, unres, ws)
    torch.cuda.synchronize()
    want = od.dedup_map(od.leaf_digests(buf, slab))
    assert int(unres.item()) == 0
    assert np.array_equal(fi.cpu().numpy(), want)
    # second call on the same workspace (it clears its own table) with fewer leaves
    kvg.kvg_dedup_map(torch.from_numpy(dg[:100]).cuda(), 100, fi, unres, ws)
    torch.cuda.synchronize()
    assert np.array_equal(fi[:100].cpu().numpy(), want[:100]) and int(unres.item()) == 0


def test_artifact_digests_equal_restored_pages(kvg):
    """Content addresses survive the round trip: the slabs of a deposited artifact and of a
    re-deposit of the pages it was grafted into have the same digests and Merkle root."""
    from paper_2607_14431_amd import harness as h
    from synth.workloads import BLOCK12B, scaled
    w = scaled(BLOCK12B, n_layers=4, prefix=1024, suffix=16, decode_steps=1)
    src = h.new_arm(w, [0], w.ctx_final, seed=61, poison_id=0)
    h.fresh_prefix(src, append_only=True)
    hdr, art = h.deposit(src, 0, 0, w.prefix, 0)
    dst = h.new_arm(w, [0], w.ctx_final, seed=62, poison_id=1)
    h.graft(dst, 0, hdr, art, 0, 0)
    _, again = h.deposit(dst, 0, 0, w.prefix, 0)
    slab = w.page_size * w.head_dim * w.elem_bytes                # one (layer, K/V, page, head)
    n = art.numel() // slab
    d1 = torch.empty((n, 32), dtype=torch.uint8, device="cuda")
    d2 = torch.empty_like(d1)
    kvg.kvg_leaf_digests(art, slab, d1)
    kvg.kvg_leaf_digests(again, slab, d2)
    ws = torch.empty(kvg.kvg_merkle_workspace_bytes(n), dtype=torch.uint8, device="cuda")
    r1 = torch.zeros(32, dtype=torch.uint8, device="cuda")
    r2 = torch.zeros_like(r1)
    kvg.kvg_merkle_root(d1, n, r1, ws)
    kvg.kvg_merkle_root(d2, n, r2, ws)
    torch.cuda.synchronize()
    assert torch.equal(d1, d2) and torch.equal(r1, r2)
    host = art.cpu().numpy()
    for i in (0, n // 3, n - 1):                                   # sampled leaves against hashlib
        assert d1[i].cpu().numpy().tobytes() == hashlib.sha256(host[i * slab:(i + 1) * slab].tobytes()).digest()
    assert r1.cpu().numpy().tobytes() == od.merkle_root(d1.cpu().numpy())
