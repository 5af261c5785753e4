"""GPU parity of each kernel family against the oracle, through the C ABI.

Inputs are generated on the host (numpy generator or seeded numpy bytes) and uploaded,
or generated on the device by the input generator whose bits are checked against the
numpy side first.  No expected value comes from the GPU path.
"""

import numpy as np
import pytest
import torch

from oracle.numerics import bits_to_values
from oracle.paging import PagedPool, append_kv, deposit as o_deposit, graft as o_graft, relocate_payload
from oracle.path import expected_rows
from synth import ROLE_K, ROLE_Q, ROLE_V, normal_tensor
from synth.philox import Stream
from synth.workloads import BLOCK12B, RELOC31B, TINY, raw_rows, scaled

from gpu_helpers import (INT_VIEW, NP_BITS, RAW_DTYPE, TORCH_DTYPE, assert_rotated_close, attention_close,
                         bits_to_device, device_to_bits, pair_norm)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kvg():
    from paper_2607_14431_amd import kvg as k
    return k


@pytest.fixture(scope="module")
def harness():
    from paper_2607_14431_amd import harness as h
    return h


# --------------------------------------------------------------------------- generator
@pytest.mark.parametrize("w", [TINY, scaled(BLOCK12B, n_layers=3), scaled(RELOC31B, n_layers=2)])
def test_device_generator_matches_numpy(w):
    from synth.gpu import raw_chunk
    for role in (ROLE_Q, ROLE_K, ROLE_V):
        got = device_to_bits(raw_chunk(w, role, [0, 3], 100, 37))
        for bi, s in enumerate([0, 3]):
            want = raw_rows(w, role, s, range(w.n_layers), 100, 37)
            assert np.array_equal(got[:, bi], want)


def test_device_generator_store_needles():
    """Store blocks with needles: the device generator plants the same needle rows as numpy,
    for a chunk holding the needle and for the window view the large store decodes over."""
    import dataclasses
    from synth.gpu import raw_chunk
    from synth.workloads import STORE12B, STORE_UNIT
    w = dataclasses.replace(STORE12B, n_layers=2)
    for b in (0, 81, w.store_blocks - 1):
        t = w.needle_offset(b)
        blk = dataclasses.replace(w, blocks_per_seq=1, block_tokens=0, prefix=4096, suffix=0, decode_steps=0,
                                  batch=1, fixed_unit=STORE_UNIT + b)
        lo = max(0, t - 20)
        for role in (ROLE_K, ROLE_V):
            got = device_to_bits(raw_chunk(blk, role, [0], lo, 41))
            assert np.array_equal(got[:, 0], raw_rows(blk, role, 0, range(2), lo, 41))
    # a window whose slot 1 holds block 81 (own position 4096), then a sequence's own tokens
    view = dataclasses.replace(w, prefix=8192, blocks_per_seq=1, block_tokens=0,
                               explicit_segments=((0, 4096, STORE_UNIT + 8, 0), (4096, 4096, STORE_UNIT + 81, 0)))
    t = 4096 + w.needle_offset(81)
    got = device_to_bits(raw_chunk(view, ROLE_K, [0, 5], t - 3, 40))
    for bi, s in enumerate([0, 5]):
        assert np.array_equal(got[:, bi], raw_rows(view, ROLE_K, s, range(2), t - 3, 40))


# --------------------------------------------------------------------------- append
@pytest.mark.parametrize("dtype,D,pairing", [("bf16", 256, 0), ("bf16", 128, 1), ("f32", 64, 0), ("f32", 64, 1),
                                             ("bf16", 64, 0), ("fp8", 256, 0), ("fp8", 128, 1), ("fp8", 64, 0)])
def test_append_matches_oracle(kvg, dtype, D, pairing):
    L, Hq, Hkv, B, chunk, max_pages = 2, 4, 2, 3, 37, 12
    n_pages = 48
    raw = RAW_DTYPE[dtype]
    poison = 0x7F if dtype == "fp8" else 0x7FC1
    rng = np.random.default_rng(D + pairing)
    tables = rng.permutation(n_pages)[: B * max_pages].reshape(B, max_pages).astype(np.int32)
    ctx = np.array([0, 19, 150], dtype=np.int32)
    start = np.array([0, 2_853_000, 8192], dtype=np.int64)
    cache = kvg.Cache.allocate(L, n_pages, Hq, Hkv, D, TORCH_DTYPE[dtype])
    cache.k_pool.view(INT_VIEW[dtype]).fill_(poison)
    cache.v_pool.view(INT_VIEW[dtype]).fill_(poison)
    st = Stream(9, ROLE_K, 1)
    sv = Stream(9, ROLE_V, 1)
    k_bits = normal_tensor(5, st, range(L), 0, B * chunk, Hkv, D, -1, raw).reshape(L, B, chunk, Hkv, D)
    v_bits = normal_tensor(5, sv, range(L), 0, B * chunk, Hkv, D, -1, raw).reshape(L, B, chunk, Hkv, D)
    seqs = kvg.Seqs(torch.from_numpy(tables).cuda(), torch.from_numpy(ctx).cuda(), torch.from_numpy(start).cuda(),
                    int(ctx.max()))
    kvg.kvg_append(cache, seqs, kvg.rope(10000.0, pairing), 0, L, chunk, bits_to_device(k_bits, raw),
                   bits_to_device(v_bits, raw))
    torch.cuda.synchronize()
    pool = PagedPool(L, n_pages, Hkv, 16, D, dtype, fill_bits=poison)
    pname = "half" if pairing == 0 else "interleaved"
    for b in range(B):
        append_kv(pool, tables[b], int(ctx[b]), k_bits[:, b], v_bits[:, b],
                  start[b] + ctx[b] + np.arange(chunk), 10000.0, pname, raw_dtype=raw)
    gk, gv = device_to_bits(cache.k_pool), device_to_bits(cache.v_pool)
    assert np.array_equal(gv, pool.v)                      # values: exact (rounded once for fp8), poison elsewhere
    written = pool.k != poison
    assert np.array_equal(gk[~written], pool.k[~written])  # untouched slots keep their poison
    kv_oracle = bits_to_values(pool.k, dtype)
    got = bits_to_values(gk, dtype)[written]
    want = kv_oracle[written]
    # rotation preserves pair norms, so the oracle's stored pair norm bounds the fp32 error
    assert_rotated_close(got, want, pair_norm(kv_oracle, pairing)[written] * 1.01, dtype)


# --------------------------------------------------------------------------- deposit / graft
@pytest.mark.parametrize("dtype,D,n_tokens", [("bf16", 256, 16 * 7), ("bf16", 128, 16 * 7 - 5), ("f32", 64, 1),
                                              ("f32", 256, 33), ("fp8", 256, 16 * 7 - 5), ("fp8", 64, 17)])
def test_deposit_and_graft_bit_exact(kvg, dtype, D, n_tokens):
    L, Hq, Hkv, n_pages = 3, 4, 2, 40
    rng = np.random.default_rng(n_tokens)
    nd = NP_BITS[dtype]
    src_bits = rng.integers(0, np.iinfo(nd).max, size=(L, n_pages, Hkv, 16, D), dtype=np.uint64).astype(nd)
    cache = kvg.Cache.allocate(L, n_pages, Hq, Hkv, D, TORCH_DTYPE[dtype])
    cache.k_pool.copy_(bits_to_device(src_bits, dtype))
    cache.v_pool.copy_(bits_to_device(src_bits[::-1].copy(), dtype))
    table = rng.permutation(n_pages)[:10].astype(np.int32)
    first = 16 * 2
    pool = PagedPool(L, n_pages, Hkv, 16, D, dtype)
    pool.k[...] = src_bits
    pool.v[...] = src_bits[::-1]
    want = o_deposit(pool, table, first, n_tokens)
    payload = torch.empty(kvg.kvg_payload_bytes(cache, n_tokens), dtype=torch.uint8, device="cuda")
    payload.fill_(0xAB)
    kvg.kvg_deposit(cache, torch.from_numpy(table).cuda(), first, n_tokens, payload)
    torch.cuda.synchronize()
    assert np.array_equal(payload.cpu().numpy().view(nd).reshape(want.shape), want)

    # graft a seeded payload into another table of a poisoned pool
    pay_bits = rng.integers(0, np.iinfo(nd).max, size=want.shape, dtype=np.uint64).astype(nd)
    tail = n_tokens - (want.shape[2] - 1) * 16
    pay_bits[:, :, -1, :, tail:, :] = 0
    dst_table = rng.permutation(n_pages)[:10].astype(np.int32)
    poison = 0x5A if dtype == "fp8" else 0x5A5A
    cache.k_pool.view(INT_VIEW[dtype]).fill_(poison)
    cache.v_pool.view(INT_VIEW[dtype]).fill_(poison)
    hdr = kvg.kvg_artifact_header_init(cache, n_tokens, 0, kvg.rope())
    dev_payload = torch.from_numpy(pay_bits.view(np.uint8).reshape(-1)).cuda()
    kvg.kvg_graft(cache, hdr, dev_payload, torch.from_numpy(dst_table).cuda(), first, 0)
    torch.cuda.synchronize()
    opool = PagedPool(L, n_pages, Hkv, 16, D, dtype, fill_bits=poison)
    o_graft(opool, pay_bits, dst_table, first, n_tokens)
    assert np.array_equal(device_to_bits(cache.k_pool), opool.k)
    assert np.array_equal(device_to_bits(cache.v_pool), opool.v)


@pytest.mark.parametrize("dtype,D,d,pairing", [("bf16", 128, 8192, 0), ("bf16", 256, -4096, 0),
                                               ("bf16", 128, 8192, 1), ("f32", 64, 2_850_000, 0),
                                               ("f32", 64, 8192, 1), ("fp8", 128, 8192, 0), ("fp8", 64, -300, 0),
                                               ("fp8", 128, 8192, 1)])
def test_relocated_graft_matches_oracle(kvg, dtype, D, d, pairing):
    L, Hq, Hkv, n_tokens, n_pages = 2, 4, 2, 16 * 5 - 3, 16
    st = Stream(11, ROLE_K, 0)
    if dtype == "fp8":       # a stored fp8 block: bf16 values rounded once
        from oracle.numerics import fp8_values_to_bits, round_fp8
        raw = normal_tensor(3, st, range(L), 0, 2 * 5 * 16, Hkv, D, -1, "bf16")
        kb = fp8_values_to_bits(round_fp8(bits_to_values(raw, "bf16"))).reshape(L, 2, 5, 16, Hkv, D)
    else:
        kb = normal_tensor(3, st, range(L), 0, 2 * 5 * 16, Hkv, D, -1, dtype).reshape(L, 2, 5, 16, Hkv, D)
    pay = np.ascontiguousarray(np.moveaxis(kb, 4, 3))           # [L][2][pages][Hkv][16][D]
    pay[:, :, -1, :, 13:, :] = 0
    cache = kvg.Cache.allocate(L, n_pages, Hq, Hkv, D, TORCH_DTYPE[dtype])
    poison = {"fp8": 0x7F, "bf16": 0x7FC1, "f32": 0x7FC00001}[dtype]
    cache.k_pool.view(INT_VIEW[dtype]).fill_(poison)              # every slot the graft must not touch
    cache.v_pool.view(INT_VIEW[dtype]).fill_(poison)
    own = 1000
    hdr = kvg.kvg_artifact_header_init(cache, n_tokens, own, kvg.rope(10000.0, pairing))
    table = np.array([9, 3, 14, 0, 7], dtype=np.int32)
    dev = torch.from_numpy(pay.view(np.uint8).reshape(-1)).cuda()
    with pytest.raises(kvg.KvgError) as e:
        kvg.kvg_graft(cache, hdr, dev, torch.from_numpy(table).cuda(), 0, own + d)
    assert e.value.name == "KVG_E_POSITION"
    kvg.kvg_graft(cache, hdr, dev, torch.from_numpy(table).cuda(), 0, own + d, kvg.KVG_GRAFT_ALLOW_RELOCATE)
    torch.cuda.synchronize()
    want = relocate_payload(pay, n_tokens, d, 10000.0, dtype, ("half", "interleaved")[pairing])
    gk = device_to_bits(cache.k_pool)[:, table]                 # [L][pages][Hkv][16][D]
    gv = device_to_bits(cache.v_pool)[:, table]
    valid = np.zeros((5, 16), dtype=bool)
    valid.reshape(-1)[:n_tokens] = True
    sel = valid[None, :, None, :, None].repeat(L, 0).repeat(Hkv, 2).repeat(D, 4)
    assert np.array_equal(gv[sel], want[:, 1][sel])
    got = bits_to_values(gk, dtype)[sel]
    exp = bits_to_values(want[:, 0], dtype)[sel]
    norm = pair_norm(bits_to_values(pay[:, 0], dtype), pairing)[sel]
    assert_rotated_close(got, exp, norm, dtype)
    # the last page's rows past the block, and every page outside the table, keep their poison
    pk, pv = device_to_bits(cache.k_pool), device_to_bits(cache.v_pool)
    p_bits = np.array(poison).astype(NP_BITS[dtype])
    assert np.all(gk[~sel] == p_bits) and np.all(gv[~sel] == p_bits)
    others = np.setdiff1d(np.arange(n_pages), table)
    assert np.all(pk[:, others] == p_bits) and np.all(pv[:, others] == p_bits)


# --------------------------------------------------------------------------- attention
ATTN_CASES = [
    scaled(TINY, prefix=40, suffix=24, decode_steps=3),
    scaled(TINY, prefix=600, suffix=70, decode_steps=2, batch=2),
    scaled(BLOCK12B, n_layers=2, prefix=530, suffix=45, decode_steps=2),
    scaled(RELOC31B, n_layers=2, prefix=1030, suffix=33, decode_steps=2, start_pos=0, batch=2),
    # sliding-window layers (every third layer global)
    scaled(BLOCK12B, n_layers=3, prefix=530, suffix=45, decode_steps=2, sliding_window=300, global_every=3),
    # fp8 E4M3 caches (bf16 inputs), D 256 and D 128, one with windows
    scaled(BLOCK12B, n_layers=2, prefix=530, suffix=45, decode_steps=2, dtype="fp8"),
    scaled(RELOC31B, n_layers=2, prefix=1030, suffix=33, decode_steps=2, start_pos=0, batch=2, dtype="fp8",
           sliding_window=700, global_every=2),
]


@pytest.mark.parametrize("w", ATTN_CASES,
                         ids=lambda w: f"{w.name}-{w.dtype}-p{w.prefix}-s{w.suffix}-b{w.batch}-w{w.sliding_window}")
def test_attention_matches_oracle(harness, w):
    seqs = list(range(w.batch))
    arm = harness.new_arm(w, seqs, w.ctx_final, seed=1, poison_id=0)
    harness.fresh_prefix(arm, append_only=True)
    res = harness.continue_arm(arm)
    torch.cuda.synchronize()
    rows = list(range(w.prefix, w.ctx_final))
    for bi, s in enumerate(seqs):
        want = expected_rows(w, s, range(w.n_layers), rows)           # [L][rows][Hq][D]
        got_suf = res.suffix[:, bi].cpu().numpy().astype(np.float64)   # [L][S][Hq][D]
        got_dec = res.decode[:, :, bi].cpu().numpy().astype(np.float64)  # [steps][L][Hq][D]
        got = np.concatenate([got_suf, np.moveaxis(got_dec, 0, 1)], axis=1)
        attention_close(got, want, w.dtype)
