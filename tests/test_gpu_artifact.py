"""A deposited block as a file, restored elsewhere (cross-context restore, Sec. 3.2; block
digests, Sec. 4.11): deposit, seal (the library's Merkle root of the payload's page-slab
leaves, checked against the oracle's), write header + payload to a file, free the writer's
cache and payload, read the file back into host-pinned memory, verify the digest, graft into
a fresh cache with another page permutation and poison, and run the suffix and decode steps:
the outputs equal the writer's fresh computation byte for byte and the restored pages
re-deposit to the file's payload.  A flipped payload byte or an inconsistent header field is
rejected with KVG_E_CORRUPT."""

import gc
import hashlib

import numpy as np
import pytest
import torch

from oracle.digest import leaf_digests, merkle_root
from synth.workloads import BLOCK12B, scaled

pytestmark = pytest.mark.gpu

CASES = [
    # workload, compare the digest with the oracle's
    (scaled(BLOCK12B, n_layers=6, prefix=1000, suffix=40, decode_steps=3), True),   # ragged last page
    (BLOCK12B, True),                                                                # the full 1.5 GiB block
]


@pytest.mark.parametrize("w,oracle_root", CASES, ids=["12b-6layers-1000tok", "12b-block4096"])
def test_artifact_file_round_trip(tmp_path, w, oracle_root):
    from paper_2607_14431_amd import harness as h, kvg
    path = str(tmp_path / "block.kvga")
    print(f"{w.name} {w.n_layers} layers, {w.prefix} tokens: writer", flush=True)
    fresh = h.new_arm(w, [0], w.ctx_final, seed=300, poison_id=0)
    h.fresh_prefix(fresh)
    hdr, payload = h.deposit(fresh, 0, 0, w.prefix, 0)
    ws = h.artifact_workspace(hdr)
    kvg.kvg_artifact_seal(hdr, payload, ws)
    leaf = w.page_size * w.head_dim * w.elem_bytes
    assert hdr.digest_leaf_bytes == leaf and bytes(hdr.digest) != bytes(32)
    host_payload = payload.cpu().numpy()
    if oracle_root:
        assert bytes(hdr.digest) == merkle_root(leaf_digests(host_payload, leaf)), "digest differs from the oracle's"
    file_sha = hashlib.sha256(host_payload.tobytes()).hexdigest()
    want = h.continue_arm(fresh).digest()
    h.save_artifact(path, hdr, payload)
    del fresh, payload, host_payload
    gc.collect()
    torch.cuda.empty_cache()

    print("reader: load, verify, graft into a fresh cache", flush=True)
    hdr2, pinned = h.load_artifact(path)
    assert bytes(hdr2) == bytes(hdr)
    assert kvg.kvg_artifact_verify(hdr2, pinned, ws) == 0
    g = h.new_arm(w, [0], w.ctx_final, seed=400, poison_id=1, spare_pages=3)
    h.graft(g, 0, hdr2, pinned, 0, 0)                    # the kernel reads the pinned payload
    _, restored = h.deposit(g, 0, 0, w.prefix, 0)
    assert kvg.kvg_artifact_verify(hdr2, restored, ws) == 0
    assert hashlib.sha256(restored.cpu().numpy().tobytes()).hexdigest() == file_sha
    assert h.continue_arm(g).digest() == want, "graft from the file != fresh"

    print("reader: corrupted payload and header", flush=True)
    host = pinned.host.numpy()
    for off in (0, hdr2.payload_bytes // 2 + 12345, hdr2.payload_bytes - 1):
        host[off] ^= 0x10
        assert kvg.kvg_artifact_verify(hdr2, pinned, ws) == -7, f"flipped byte {off} not detected"
        host[off] ^= 0x10
    assert kvg.kvg_artifact_verify(hdr2, pinned, ws) == 0
    bad = kvg.kvg_artifact_hdr.from_buffer_copy(bytes(hdr2))
    bad.n_tokens += 20                                    # geometry no longer matches the payload size
    assert kvg.kvg_artifact_verify(bad, pinned, ws) == -7
    with pytest.raises(kvg.KvgError) as e:
        h.graft(g, 0, bad, pinned, 0, 0)
    assert e.value.status == -7
    bad = kvg.kvg_artifact_hdr.from_buffer_copy(bytes(hdr2))
    bad.digest[5] ^= 1                                    # a header whose digest was altered
    assert kvg.kvg_artifact_verify(bad, pinned, ws) == -7
    del g, pinned, restored
    gc.collect()
    torch.cuda.empty_cache()
