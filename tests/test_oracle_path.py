"""The oracle's end-to-end fresh path agrees with the paged deposit/graft route."""

import numpy as np
import pytest

from oracle.attention import attend_paged
from oracle.numerics import bits_to_values
from oracle.paging import PagedPool, append_kv, deposit, graft, relocate_payload
from oracle.path import expected_rows, fresh_kv, relocated_kv
from synth.workloads import ROLE_K, ROLE_V, TINY, RELOC31B, raw_rows, scaled

W = scaled(TINY, prefix=48, suffix=8, decode_steps=3)
W8 = scaled(TINY, dtype="fp8", sigma_log2=-1, prefix=48, suffix=8, decode_steps=3)   # bf16 in, fp8 stored
FILL = {"f32": 0xFFFFFFFF, "bf16": 0xFFFF, "fp8": 0xFF}


def _paged_fresh(w, table, start_pos, n):
    pool = PagedPool(w.n_layers, 32, w.n_kv_heads, w.page_size, w.head_dim, w.dtype, fill_bits=FILL[w.dtype])
    k = raw_rows(w, ROLE_K, 0, range(w.n_layers), 0, n)
    v = raw_rows(w, ROLE_V, 0, range(w.n_layers), 0, n)
    # chunked like the GPU path: prefix, then suffix, then one token at a time
    cuts = [0, w.prefix, w.prefix + w.suffix] + list(range(w.prefix + w.suffix + 1, n + 1))
    for a, b in zip(cuts[:-1], cuts[1:]):
        append_kv(pool, table, a, k[:, a:b], v[:, a:b], start_pos + np.arange(a, b), w.rope_base,
                  raw_dtype=w.raw_dtype)
    return pool


@pytest.mark.parametrize("W", [W, W8], ids=["f32", "fp8"])
def test_graft_route_equals_fresh_definition(W):
    n = W.ctx_final
    rows = np.arange(W.prefix, n)
    t_fresh = list(np.random.default_rng(0).permutation(32)[:4])
    t_graft = list(np.random.default_rng(1).permutation(32)[:4])
    fresh_pool = _paged_fresh(W, t_fresh, 0, n)
    payload = deposit(fresh_pool, t_fresh, 0, W.prefix)
    graft_pool = PagedPool(W.n_layers, 32, W.n_kv_heads, W.page_size, W.head_dim, W.dtype)
    graft(graft_pool, payload, t_graft, 0, W.prefix)
    k = raw_rows(W, ROLE_K, 0, [0], 0, n)
    v = raw_rows(W, ROLE_V, 0, [0], 0, n)
    append_kv(graft_pool, t_graft, W.prefix, k[:, W.prefix:], v[:, W.prefix:],
              np.arange(W.prefix, n), W.rope_base, raw_dtype=W.raw_dtype)
    want = expected_rows(W, 0, [0], rows)
    from oracle.path import query_rows
    q = query_rows(W, 0, [0], rows, 0)[0]
    got_fresh = attend_paged(q, rows, fresh_pool, t_fresh, n, 0, W.scale)
    got_graft = attend_paged(q, rows, graft_pool, t_graft, n, 0, W.scale)
    assert np.array_equal(got_fresh, want[0])
    assert np.array_equal(got_graft, want[0])         # Eq. 1 holds in the oracle too


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_relocated_kv_matches_payload_relocation(dtype):
    w = scaled(RELOC31B, n_layers=1, n_q_heads=4, n_kv_heads=2, prefix=32, suffix=8, decode_steps=0, dtype=dtype)
    n = w.prefix + w.suffix
    table = [0, 1, 2]
    pool = _paged_fresh(scaled(w, decode_steps=0, suffix=0, prefix=32), table[:2], w.own_pos, 32)
    payload = deposit(pool, table[:2], 0, 32)
    moved = relocate_payload(payload, 32, w.start_pos - w.own_pos, w.rope_base, w.dtype)
    k_rel, v_rel = relocated_kv(w, 0, [0], 32, n)
    tgt = PagedPool(1, 4, w.n_kv_heads, w.page_size, w.head_dim, w.dtype)
    graft(tgt, moved, table, 0, 32)
    kb, vb = tgt.read_tokens(table, 0, 32)
    assert np.array_equal(bits_to_values(kb[0], w.dtype), k_rel[0, :32])
    assert np.array_equal(bits_to_values(vb[0], w.dtype), v_rel[0, :32])
    # tokens after the block are fresh at the new offset
    k_new, _ = fresh_kv(w, 0, [0], n, w.start_pos)
    assert np.array_equal(k_rel[0, 32:], k_new[0, 32:])


def test_fp8_cache_holds_rounded_values():
    """An fp8 cache stores the bf16 inputs rounded once to E4M3: values exactly, keys after
    the fp64 rotation; both are on the fp8 grid and within half a grid step of the input."""
    from oracle.numerics import round_fp8
    n = 40
    k, v = fresh_kv(W8, 0, [0], n, 0)
    v_raw = bits_to_values(raw_rows(W8, ROLE_V, 0, [0], 0, n), "bf16")
    assert np.array_equal(round_fp8(k), k) and np.array_equal(round_fp8(v), v)
    assert np.array_equal(v, round_fp8(v_raw))
    step = np.where(np.abs(v_raw) >= 2.0 ** -6, np.ldexp(1.0, np.frexp(np.abs(v_raw))[1] - 4), 2.0 ** -9)
    assert np.all(np.abs(v - v_raw) <= step / 2)
    assert np.any(v != v_raw)                              # the rounding is not vacuous


def test_query_rows_on_scattered_rows():
    """query_rows over a sorted, non-contiguous row list (as the full-size tests sample rows)
    equals rotating each row's raw query alone, and the runs it cuts the list into are the
    maximal contiguous ones."""
    from oracle.path import _runs, query_rows
    from oracle.rope import rotate
    from synth.workloads import ROLE_Q
    assert _runs(np.array([3, 4, 9, 17, 18, 19, 40])) == [(3, 5), (9, 10), (17, 20), (40, 41)]
    assert _runs(np.array([7])) == [(7, 8)]
    assert _runs(np.arange(5, 12)) == [(5, 12)]
    w = scaled(TINY, n_layers=2, prefix=48, suffix=8, decode_steps=3)
    rows = [0, 1, 5, 17, 18, 19, 40, 58]
    start = 37
    got = query_rows(w, 0, [0, 1], rows, start)
    assert got.shape == (2, len(rows), w.n_q_heads, w.head_dim)
    for i, r in enumerate(rows):
        q = bits_to_values(raw_rows(w, ROLE_Q, 0, [0, 1], r, 1), w.raw_dtype)
        want = rotate(q, np.array([start + r], dtype=np.float64), w.rope_base)
        assert np.array_equal(got[:, i], want[:, 0])


def test_expected_rows_subset_of_contiguous():
    """expected_rows on an unsorted scattered list returns, in ascending row order, the rows of
    the contiguous computation over the same keys (equal up to the fp64 summation order of
    the matrix products, which depends on how many rows are computed together)."""
    w = scaled(TINY, prefix=48, suffix=8, decode_steps=3)
    rows = [40, 3, 17, 18, 9]
    full = expected_rows(w, 0, [0], range(0, 41))
    part = expected_rows(w, 0, [0], rows)
    assert np.abs(part[0] - full[0][sorted(rows)]).max() <= 1e-13
    # a permuted or shifted row would differ by the outputs' own size (~0.1), not 1e-13
    assert np.abs(part[0] - full[0][rows]).max() > 1e-3
