"""Pins for the oracle's paged pool, deposit (capture) and graft (restore)."""

import hashlib

import numpy as np
import pytest

from oracle.attention import attend, attend_paged
from oracle.numerics import bits_to_values, round_bf16
from oracle.paging import PagedPool, append_kv, deposit, graft, relocate_payload
from oracle.rope import rotate
from synth import f32_to_bf16_bits

rng = np.random.default_rng(23)
L, HKV, P, D = 2, 2, 16, 32


def _bits(shape, scale=0.5):
    return f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def _filled_pool(n_tokens, table, n_pages=64, fill=0xFFFF):
    pool = PagedPool(L, n_pages, HKV, P, D, "bf16", fill_bits=fill)
    pool.write_tokens(table, 0, _bits((L, n_tokens, HKV, D)), _bits((L, n_tokens, HKV, D)))
    return pool


def test_sha256_vectors():
    # FIPS 180-4 example digests, for the digest used on payloads
    assert hashlib.sha256(b"abc").hexdigest() == \
        "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"
    assert hashlib.sha256(b"").hexdigest() == \
        "e3b0c44298fc1c149afbf4c8996fb92427ae41e4649b934ca495991b7852b855"


@pytest.mark.parametrize("n_tokens", [16 * 5, 16 * 5 - 3, 1])
def test_deposit_graft_round_trip(n_tokens):
    src_table = list(rng.permutation(64)[:8])
    dst_table = list(rng.permutation(64)[:8])
    src = _filled_pool(n_tokens, src_table)
    payload = deposit(src, src_table, 0, n_tokens)
    dst = PagedPool(L, 64, HKV, P, D, "bf16", fill_bits=0x7FC1)
    graft(dst, payload, dst_table, 0, n_tokens)
    ks, vs = src.read_tokens(src_table, 0, n_tokens)
    kd, vd = dst.read_tokens(dst_table, 0, n_tokens)
    assert np.array_equal(ks, kd) and np.array_equal(vs, vd)
    # restored pages re-deposit to the identical artifact
    again = deposit(dst, dst_table, 0, n_tokens)
    assert hashlib.sha256(again.tobytes()).digest() == hashlib.sha256(payload.tobytes()).digest()
    # zero tail in the last payload page; rows past the block untouched in the target
    rows = n_tokens - (payload.shape[2] - 1) * P
    assert not payload[:, :, -1, :, rows:, :].any()
    last = dst_table[(n_tokens - 1) // P]
    assert np.all(dst.k[:, last, :, rows:, :] == 0x7FC1)


def test_deposit_layout_is_layer_kv_page_head_row():
    table = [5, 2, 9]
    pool = _filled_pool(48, table)
    payload = deposit(pool, table, 0, 48)
    assert payload.shape == (L, 2, 3, HKV, P, D)
    assert np.array_equal(payload[1, 0, 2, 1, 7], pool.k[1, 9, 1, 7])
    assert np.array_equal(payload[0, 1, 1, 0, 3], pool.v[0, 2, 0, 3])


def test_graft_at_page_aligned_offset():
    table = list(range(10, 20))
    src = _filled_pool(32, [0, 1])
    payload = deposit(src, [0, 1], 0, 32)
    dst = PagedPool(L, 64, HKV, P, D, "bf16")
    graft(dst, payload, table, 48, 32)
    assert np.array_equal(dst.k[:, 13], src.k[:, 0]) and np.array_equal(dst.v[:, 14], src.v[:, 1])
    with pytest.raises(ValueError):
        graft(dst, payload, table, 8, 32)


def test_attention_independent_of_physical_pages():
    n = 70
    k_bits, v_bits = _bits((L, n, HKV, D)), _bits((L, n, HKV, D))
    t1 = list(range(5))
    t2 = list(rng.permutation(40)[:5])
    p1 = PagedPool(L, 40, HKV, P, D, "bf16")
    p2 = PagedPool(L, 40, HKV, P, D, "bf16", fill_bits=0x1234)
    p1.write_tokens(t1, 0, k_bits, v_bits)
    p2.write_tokens(t2, 0, k_bits, v_bits)
    q = rng.standard_normal((3, 4, D))
    idx = np.array([10, 40, 69])
    o1 = attend_paged(q, idx, p1, t1, n, 1, 0.2)
    o2 = attend_paged(q, idx, p2, t2, n, 1, 0.2)
    assert np.array_equal(o1, o2)
    dense = attend(q, idx, bits_to_values(k_bits[1], "bf16"), bits_to_values(v_bits[1], "bf16"), 0.2)
    assert np.array_equal(o1, dense)


def test_append_rotates_and_rounds():
    table = [3, 1]
    pool = PagedPool(1, 4, HKV, P, D, "bf16")
    k_raw, v_raw = _bits((1, 20, HKV, D)), _bits((1, 20, HKV, D))
    append_kv(pool, table, 0, k_raw, v_raw, np.arange(100, 120), 1e4)
    k_st, v_st = pool.read_tokens(table, 0, 20)
    want = round_bf16(rotate(bits_to_values(k_raw, "bf16"), np.arange(100, 120), 1e4))
    assert np.array_equal(bits_to_values(k_st, "bf16"), want)
    assert np.array_equal(v_st, v_raw)


def test_relocate_zero_is_identity_and_round_trip():
    table = [0, 1, 2]
    pool = _filled_pool(40, table)
    payload = deposit(pool, table, 0, 40)
    assert np.array_equal(relocate_payload(payload, 40, 0, 1e4, "bf16"), payload)
    moved = relocate_payload(payload, 40, 8192, 1e4, "bf16")
    assert np.array_equal(moved[:, 1], payload[:, 1])                 # V untouched
    back = relocate_payload(moved, 40, -8192, 1e4, "bf16")
    a = bits_to_values(back[:, 0], "bf16")
    b = bits_to_values(payload[:, 0], "bf16")
    # each rounding errs by half an ulp of a value no larger than the pair's norm r
    # (half-split pairs i, i + D/2), and rotation preserves the error's norm
    r = np.sqrt(b[..., : D // 2] ** 2 + b[..., D // 2:] ** 2)
    r = np.concatenate([r, r], axis=-1)
    ulp_r = np.ldexp(1.0, np.frexp(np.maximum(r, 1e-30))[1] - 8)
    assert np.all(np.abs(a - b) <= 1.5 * ulp_r)
    assert np.any(a != b)                                              # not byte-exact
    assert not moved[:, 0, -1, :, 8:, :].any()                          # tail stays zero
