"""Seeded input generator: known-answer vectors, distribution, bf16 rounding."""

import os

import numpy as np
import pytest

from synth import f32_to_bf16_bits, bf16_bits_to_f32, normal_f32, normal_tensor, philox4x32_10
from synth.philox import Stream, TOKEN_STRIDE
from synth.workloads import WORKLOADS, WINDOW12B, raw_rows, ROLE_K

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            rows.append([int(x, 16) for x in line.split()])
    return rows


@pytest.mark.parametrize("row", _kat())
def test_philox_known_answers(row):
    ctr = np.array([row[:4]], dtype=np.uint32)
    out = philox4x32_10(ctr, (row[4], row[5]))[0]
    assert [int(x) for x in out] == row[6:]


def test_normal_moments_and_range():
    v = normal_f32(7, 3, np.arange(400_000, dtype=np.uint64), 0).astype(np.float64)
    assert abs(v.mean()) < 0.01
    assert abs(v.std() - 1.0) < 0.01
    assert np.abs(v).max() <= 6138 / 1024
    # exactness: every value is an integer multiple of 2**-10
    assert np.all(np.ldexp(v, 10) == np.rint(np.ldexp(v, 10)))
    half = normal_f32(7, 3, np.arange(1000, dtype=np.uint64), -1)
    assert np.array_equal(half * 2, normal_f32(7, 3, np.arange(1000, dtype=np.uint64), 0))


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    x = normal_f32(11, 5, np.arange(100_000, dtype=np.uint64), -1)
    ties = np.array([1 + 2**-8, 1 + 3 * 2**-8, -(1 + 2**-8), 3.0, 0.0, 1e-3], dtype=np.float32)
    x = np.concatenate([x, ties])
    ours = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert bf16_bits_to_f32(f32_to_bf16_bits(np.float32([1 + 2**-8])))[0] == 1.0


def test_chunking_does_not_change_values():
    st = Stream(9, ROLE_K, 4)
    full = normal_tensor(1, st, [0, 3], 0, 40, 2, 8, -1, "bf16")
    a = normal_tensor(1, st, [0, 3], 0, 17, 2, 8, -1, "bf16")
    b = normal_tensor(1, st, [0, 3], 17, 23, 2, 8, -1, "bf16")
    assert np.array_equal(full, np.concatenate([a, b], axis=1))
    one = normal_tensor(1, st, [3], 5, 1, 2, 8, -1, "bf16")
    assert np.array_equal(one[0, 0], full[1, 5])


def test_streams_differ():
    a = normal_tensor(1, Stream(2, 2, 0), [0], 0, 4, 1, 8, 0, "f32")
    b = normal_tensor(1, Stream(2, 3, 0), [0], 0, 4, 1, 8, 0, "f32")
    assert not np.array_equal(a, b)


def test_workload_segments_cover_sequence():
    for w in WORKLOADS.values():
        if w.wid == 5:
            continue
        segs = w.segments(0)
        t = 0
        for (a, n, _, _) in segs:
            assert a == t
            t += n
        assert t == w.ctx_final
    # window slots draw blocks whose own position matches the slot
    for s in range(3):
        for j in range(WINDOW12B.blocks_per_seq):
            assert WINDOW12B.seq_block(s, j) % WINDOW12B.blocks_per_seq == j
    assert TOKEN_STRIDE > WORKLOADS[5].store_tokens


def test_raw_rows_uses_store_blocks():
    w = WINDOW12B
    b1 = w.seq_block(0, 1)
    r = raw_rows(w, ROLE_K, 0, [0], 4096 + 5, 3)
    from synth.workloads import STORE_UNIT
    direct = normal_tensor(w.seed, w.stream(ROLE_K, STORE_UNIT + b1), [0], 5, 3, w.n_kv_heads,
                           w.head_dim, w.sigma_log2, "bf16")
    assert np.array_equal(r, direct)


def test_store_needles():
    """Every store block of the large store carries its needle inside its own tokens (the last,
    partial block included); the needle token's K and V rows come from the needle streams and
    every other row is the block's ordinary stream; a range without the needle is untouched."""
    import dataclasses
    from synth.workloads import ROLE_Q, ROLE_V, STORE12B, STORE_UNIT, needle_row
    w = STORE12B
    last = w.store_blocks - 1
    assert w.needle_span == w.store_block_tokens(last)
    offs = [w.needle_offset(b) for b in range(w.store_blocks)]
    assert all(0 <= t < w.store_block_tokens(b) for b, t in zip(range(w.store_blocks), offs))
    assert len(set(offs)) > 500                     # seeded, not constant
    b = 81
    t = w.needle_offset(b)
    blk = dataclasses.replace(w, n_layers=2, blocks_per_seq=1, block_tokens=0, prefix=4096, suffix=0,
                              decode_steps=0, batch=1, fixed_unit=STORE_UNIT + b)
    lo = max(0, t - 3)
    for role in (ROLE_K, ROLE_V):
        got = raw_rows(blk, role, 0, [0, 1], lo, 7)
        plain = normal_tensor(w.seed, w.stream(role, STORE_UNIT + b), [0, 1], lo, 7, w.n_kv_heads, w.head_dim,
                              w.sigma_log2, "bf16")
        needle = needle_row(w, role, STORE_UNIT + b, [0, 1])
        assert np.array_equal(got[:, t - lo], needle[:, 0])
        keep = [i for i in range(7) if i != t - lo]
        assert np.array_equal(got[:, keep], plain[:, keep])
        assert not np.array_equal(needle[:, 0], plain[:, t - lo])
    q = raw_rows(blk, ROLE_Q, 0, [0], lo, 7)        # queries carry no needle
    assert np.array_equal(q, normal_tensor(w.seed, w.stream(ROLE_Q, STORE_UNIT + b), [0], lo, 7, w.n_q_heads,
                                           w.head_dim, w.sigma_log2, "bf16"))
    other = raw_rows(blk, ROLE_K, 0, [0], t + 1, 5) if t + 6 <= 4096 else raw_rows(blk, ROLE_K, 0, [0], 0, 5)
    assert other.shape[1] == 5
    # workloads without needles are unchanged
    assert WINDOW12B.needle_at(STORE_UNIT + 3, 0, 4096) is None
