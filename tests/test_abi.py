"""The C-ABI library loads, exports every symbol include/kvg.h declares, and validates
arguments on the host (status codes returned before any launch; no GPU needed)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvg.h")

kvg = pytest.importorskip("paper_2607_14431_amd.kvg", reason="libkvg.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvg_[a-z0-9_]+)\s*\(", text)))


def test_header_and_binding_agree():
    decl = declared_functions()
    assert decl, "no declarations parsed"
    assert sorted(kvg.EXPORTED) == decl


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(kvg.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version_and_status_strings():
    assert "gfx950" in kvg.kvg_version()
    for code in kvg.STATUS:
        assert kvg.kvg_status_str(code) != "unknown status"
    assert kvg.kvg_status_str(12345) == "unknown status"


def _cache(**kw):
    args = dict(n_layers=2, n_q_heads=4, n_kv_heads=2, head_dim=64, page_size=16, dtype=kvg.KVG_BF16,
                n_pages=8, k_pool=0x1000, v_pool=0x2000)
    args.update(kw)
    return kvg.kvg_cache(**args)


def _seqs(**kw):
    args = dict(batch=1, max_pages=4, max_ctx_len=32, shared_tokens=0, block_tables=0x3000, ctx_lens=0x4000,
                start_pos=0x5000)
    args.update(kw)
    return kvg.kvg_seqs(**args)


R = ctypes.byref


def _append(cache, seqs, chunk=8, rope=None, k=0x6000, v=0x7000, layer0=0, n_layers=2):
    rope = rope or kvg.rope()
    return kvg.raw_call("kvg_append", R(cache), R(seqs), R(rope), layer0, n_layers, chunk, ctypes.c_void_p(k),
                        ctypes.c_void_p(v), None)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), -2), (dict(page_size=32), -2), (dict(n_q_heads=6), -2), (dict(n_q_heads=32, n_kv_heads=2), -2),
    (dict(dtype=7), -3), (dict(k_pool=0), -1), (dict(n_pages=0), -2),
])
def test_append_rejects_bad_cache(kw, status):
    assert _append(_cache(**kw), _seqs()) == status


def test_append_rejects_bad_seqs_and_args():
    assert _append(_cache(), _seqs(max_ctx_len=60), chunk=8) == -5          # 68 > 4 pages * 16
    assert _append(_cache(), _seqs(block_tables=0)) == -1
    assert _append(_cache(), _seqs(shared_tokens=-1)) == -1
    assert _append(_cache(), _seqs(shared_tokens=4 * 16 + 1)) == -1      # beyond the table rows
    assert _append(_cache(), _seqs(), chunk=0) == -1
    assert _append(_cache(), _seqs(), k=0) == -1
    assert _append(_cache(), _seqs(), layer0=1, n_layers=2) == -2
    assert _append(_cache(), _seqs(), rope=kvg.kvg_rope(-1.0, 0, 0)) == -1
    assert _append(_cache(), _seqs(), rope=kvg.kvg_rope(1e4, 5, 0)) == -1


def test_payload_bytes_and_header():
    c = _cache()
    # 2 layers * (K, V) * 2 pages * 2 heads * 16 rows * 64 * 2 bytes
    assert kvg.raw_call("kvg_payload_bytes", R(c), 17) == 2 * 2 * 2 * 2 * 16 * 64 * 2
    assert kvg.raw_call("kvg_payload_bytes", R(c), 0) == 0
    hdr = kvg.kvg_artifact_hdr()
    assert kvg.raw_call("kvg_artifact_header_init", R(c), 17, 128, R(kvg.rope()), R(hdr)) == 0
    assert hdr.magic == kvg.KVG_ARTIFACT_MAGIC and hdr.version == 2 and hdr.n_tokens == 17
    assert hdr.digest_leaf_bytes == 0 and bytes(hdr.digest) == bytes(32)        # not sealed
    assert hdr.own_pos == 128 and hdr.payload_bytes == kvg.raw_call("kvg_payload_bytes", R(c), 17)
    assert ctypes.sizeof(kvg.kvg_artifact_hdr) == 96


def _graft(cache, hdr, table_len=4, first=0, target=None, flags=0):
    target = hdr.own_pos if target is None else target
    return kvg.raw_call("kvg_graft", R(cache), R(hdr), ctypes.c_void_p(0x8000), ctypes.c_void_p(0x9000),
                        table_len, first, target, flags, None)


def _hdr(cache, n=40, own=0):
    hdr = kvg.kvg_artifact_hdr()
    assert kvg.raw_call("kvg_artifact_header_init", R(cache), n, own, R(kvg.rope()), R(hdr)) == 0
    return hdr


def test_graft_validation():
    c = _cache()
    h = _hdr(c)
    assert _graft(c, h, target=5) == -4                       # relocation not allowed
    assert _graft(c, h, first=8) == -6                        # not page aligned
    assert _graft(c, h, table_len=2) == -5                    # 40 tokens need 3 pages
    assert _graft(c, h, first=16, table_len=3) == -5
    bad = _hdr(c)
    bad.magic = 0
    assert _graft(c, bad) == -7
    bad = _hdr(c)
    bad.payload_bytes += 2
    assert _graft(c, bad) == -7
    assert _graft(_cache(dtype=kvg.KVG_F32), _hdr(c)) == -3
    assert _graft(_cache(head_dim=128), _hdr(c)) == -2
    assert _graft(_cache(n_kv_heads=1, n_q_heads=2), _hdr(c)) == -2


def test_artifact_digest_validation():
    """Seal / verify: workspace size from the header alone, header inconsistencies and an
    unsealed header rejected as KVG_E_CORRUPT before anything is launched."""
    c = _cache()
    h = _hdr(c)                                           # 40 tokens: 3 pages, leaves of 16 x 64 bf16
    n_leaves = 2 * 2 * 3 * 2                              # layers x (K, V) x pages x heads
    assert h.payload_bytes == n_leaves * 16 * 64 * 2
    ws = kvg.raw_call("kvg_artifact_digest_workspace_bytes", R(h))
    assert ws >= n_leaves * 32 + 32
    verify = lambda hd, payload=0xA000, ws_bytes=ws: kvg.raw_call(  # noqa: E731
        "kvg_artifact_verify", R(hd), ctypes.c_void_p(payload), ctypes.c_void_p(0xB000), ws_bytes, None)
    seal = lambda hd, payload=0xA000, ws_bytes=ws: kvg.raw_call(  # noqa: E731
        "kvg_artifact_seal", R(hd), ctypes.c_void_p(payload), ctypes.c_void_p(0xB000), ws_bytes, None)
    assert verify(h) == -7                                # not sealed
    assert verify(h, payload=0) == -1 and seal(h, payload=0) == -1
    sealed = _hdr(c)
    sealed.digest_leaf_bytes = 16 * 64 * 2
    assert verify(sealed, payload=0xA008) == -6           # payload not 16-byte aligned
    assert verify(sealed, ws_bytes=ws - 1) == -9
    for field, value in (("magic", 0), ("version", 1), ("payload_bytes", h.payload_bytes + 64), ("n_tokens", 49),
                         ("dtype", 7), ("digest_leaf_bytes", 4096)):
        bad = _hdr(c)
        bad.digest_leaf_bytes = 16 * 64 * 2
        setattr(bad, field, value)
        assert verify(bad) == -7, field
        if field != "digest_leaf_bytes":
            assert seal(bad) == -7, field
            assert kvg.raw_call("kvg_artifact_digest_workspace_bytes", R(bad)) == 0, field


def test_deposit_validation():
    c = _cache()
    dep = lambda tl, first, n, payload=0xA000: kvg.raw_call(  # noqa: E731
        "kvg_deposit", R(c), ctypes.c_void_p(0x9000), tl, first, n, ctypes.c_void_p(payload), None)
    assert dep(4, 3, 16) == -6
    assert dep(2, 0, 40) == -5
    assert dep(4, 0, 0) == -1
    assert dep(4, 0, 16, payload=0) == -1


def test_attention_validation():
    c, s = _cache(), _seqs()
    ws = ctypes.c_void_p(0xB000)
    call = lambda ws_bytes, scale=0.125, rows=8: kvg.raw_call(  # noqa: E731
        "kvg_prefill_attn", R(c), R(s), R(kvg.rope()), 0, 2, rows, ctypes.c_void_p(1), ctypes.c_void_p(2),
        ctypes.c_void_p(3), scale, ctypes.c_void_p(4), ws, ws_bytes, None)
    need = kvg.raw_call("kvg_prefill_workspace_bytes", R(c), R(s), 2, 8)
    assert need > 0
    assert call(need - 1) == -9
    assert call(need, scale=0.0) == -1
    assert call(need, rows=40) == -5
    dneed = kvg.raw_call("kvg_decode_workspace_bytes", R(c), R(s), 2)
    assert 0 < dneed <= need
    assert kvg.raw_call("kvg_decode_attn", R(c), R(s), R(kvg.rope()), 0, 2, ctypes.c_void_p(1), ctypes.c_void_p(2),
                        ctypes.c_void_p(3), ctypes.c_float(0.125), ctypes.c_void_p(4), ws, dneed - 1, None) == -9


def test_digest_validation():
    P = ctypes.c_void_p
    leaf = lambda data, n, lb, out=0xC000: kvg.raw_call("kvg_leaf_digests", P(data), n, lb, P(out), None)  # noqa: E731
    assert leaf(0, 4096, 4096) == -1                 # null data
    assert leaf(0xA000, 0, 4096) == -1               # empty buffer
    assert leaf(0xA000, 4096, 100) == -1             # leaf not a multiple of 64
    assert leaf(0xA000, 4096, 0) == -1
    assert leaf(0xA008, 4096, 4096) == -6            # data not 16-byte aligned
    assert leaf(0xA000, 4096, 4096, out=0) == -1
    assert kvg.raw_call("kvg_merkle_workspace_bytes", 0) == 0
    need = kvg.raw_call("kvg_merkle_workspace_bytes", 1000)
    assert need >= 2 * 500 * 32
    root = lambda n, ws_bytes, ws=0xD000: kvg.raw_call(  # noqa: E731
        "kvg_merkle_root", P(0xA000), n, P(0xB000), P(ws), ws_bytes, None)
    assert root(0, need) == -1
    assert root(1000, need - 1) == -9
    assert root(1000, need, ws=0) == -9
    dneed = kvg.raw_call("kvg_dedup_workspace_bytes", 1000)
    assert dneed >= 2 * 2048 * 8                     # two tables of >= 2n slots
    dd = lambda n, ws_bytes, fi=0xB000: kvg.raw_call(  # noqa: E731
        "kvg_dedup_map", P(0xA000), n, P(fi), P(0xB800), P(0xD000), ws_bytes, None)
    assert dd(0, dneed) == -1
    assert dd(1000, dneed - 1) == -9
    assert dd(1000, dneed, fi=0) == -1


def test_logits_validation():
    """Argument checks of the logit entry points, taken on the host before any launch."""
    P = ctypes.c_void_p
    ws_need = kvg.raw_call("kvg_logits_workspace_bytes", 50, 4096)
    assert ws_need >= 64 * 4096 * 2 and kvg.raw_call("kvg_logits_workspace_bytes", 0, 4096) == 0

    def call(hid=0xA000, rows=50, H=4096, w=0xB000, V=1000, cap=30.0, out=0xC000, ws=0xD000, ws_bytes=ws_need):
        return kvg.raw_call("kvg_logits", P(hid), rows, H, P(w), V, ctypes.c_float(cap), P(out), P(ws), ws_bytes,
                            None)
    assert call(hid=0) == -1 and call(w=0) == -1 and call(out=0) == -1
    assert call(rows=0) == -1 and call(V=0) == -1 and call(H=0) == -1
    assert call(cap=-1.0) == -1 and call(cap=float("inf")) == -1 and call(cap=float("nan")) == -1
    assert call(H=4000) == -2                        # hidden not a multiple of 128
    assert call(hid=0xA004) == -6 and call(w=0xB008) == -6 and call(out=0xC00C) == -6
    assert call(ws=0) == -9 and call(ws_bytes=ws_need - 1) == -9
    assert call(ws=0xD008) == -6

    assert kvg.raw_call("kvg_logits_packed_bytes", 1000, 4096) == 1024 * 4096 * 2
    assert kvg.raw_call("kvg_logits_packed_bytes", 0, 4096) == 0
    pack = lambda w=0xA000, V=1000, H=4096, out=0xB000: kvg.raw_call(  # noqa: E731
        "kvg_logits_pack", P(w), V, H, P(out), None)
    assert pack(w=0) == -1 and pack(out=0) == -1 and pack(V=0) == -1 and pack(H=-128) == -1
    assert pack(H=4000) == -2 and pack(w=0xA002) == -6 and pack(out=0xB004) == -6

    def cmp(a=0xA000, b=0xB000, rows=4, V=100, kl=0xC000, ia=0xD000, ib=0xE000):
        return kvg.raw_call("kvg_logit_compare", P(a), P(b), rows, V, P(kl), P(ia), P(ib), None)
    assert cmp(a=0) == -1 and cmp(b=0) == -1 and cmp(kl=0) == -1 and cmp(ia=0) == -1 and cmp(ib=0) == -1
    assert cmp(rows=0) == -1 and cmp(V=-5) == -1


def test_prefill_workspace_with_shared_pages():
    """kvg_prefill_workspace_bytes grows by two partials per (layer, sequence, row, query head)
    exactly when the shared-page prefill runs: MFMA cache, batch >= 2, at least one whole
    512-key split shared, and a chunk shorter than the kernel's q-tile (32 x 8 / group = 128
    rows here)."""
    c = _cache()                                    # bf16, 4 query heads over 2 KV heads, head_dim 64
    def need(chunk, **kw):
        s = _seqs(**dict(dict(batch=4, max_pages=64, max_ctx_len=600), **kw))
        return kvg.raw_call("kvg_prefill_workspace_bytes", R(c), R(s), 2, chunk)
    rows = 2 * 4 * 8 * 4                            # layers x batch x chunk x query heads
    assert need(8, shared_tokens=512) - need(8) == rows * 2 * 2 * 4 + rows * 2 * 64 * 4
    assert need(8, shared_tokens=1000) == need(8, shared_tokens=512)   # one whole split either way
    assert need(8, shared_tokens=500) == need(8)                        # no whole split
    assert need(128, shared_tokens=512) == need(128)                    # a full q-tile per sequence
    assert need(127, shared_tokens=512) > need(127)
    assert need(8, shared_tokens=512, batch=1) == need(8, batch=1)      # nothing to share
    c32 = _cache(dtype=kvg.KVG_F32)
    s32 = _seqs(batch=4, max_pages=64, max_ctx_len=600, shared_tokens=512)
    s0 = _seqs(batch=4, max_pages=64, max_ctx_len=600)
    assert (kvg.raw_call("kvg_prefill_workspace_bytes", R(c32), R(s32), 2, 8)
            == kvg.raw_call("kvg_prefill_workspace_bytes", R(c32), R(s0), 2, 8))   # vector path: ignored


def test_launch_size_limits():
    """Calls whose grids would exceed 2^32 threads are rejected with KVG_E_SHAPE before
    anything is launched (the library never half-completes a call at launch time)."""
    big = _cache(n_layers=1 << 20, head_dim=256)        # 1M layers: 2^20 x 2 x pages x 16 slices workgroups
    h = kvg.kvg_artifact_hdr()
    assert kvg.raw_call("kvg_artifact_header_init", R(big), 4096, 0, R(kvg.rope()), R(h)) == 0
    assert kvg.raw_call("kvg_graft", R(big), R(h), ctypes.c_void_p(0x8000), ctypes.c_void_p(0x9000), 256, 0, 0, 0,
                        None) == -2
    assert kvg.raw_call("kvg_deposit", R(big), ctypes.c_void_p(0x9000), 256, 0, 4096, ctypes.c_void_p(0xA000),
                        None) == -2
    c = _cache()
    s = _seqs(batch=1 << 23, max_pages=4, max_ctx_len=32)    # 8M sequences: the decode grid overflows
    need = kvg.raw_call("kvg_decode_workspace_bytes", R(c), R(s), 2)
    assert kvg.raw_call("kvg_decode_attn", R(c), R(s), R(kvg.rope()), 0, 2, ctypes.c_void_p(1), ctypes.c_void_p(2),
                        ctypes.c_void_p(3), ctypes.c_float(0.125), ctypes.c_void_p(4), ctypes.c_void_p(0xB000), need,
                        None) == -2
    s2 = _seqs(batch=1 << 23, max_pages=4, max_ctx_len=16)   # 8M sequences x 2 tokens: 2^32 threads
    assert kvg.raw_call("kvg_append", R(c), R(s2), R(kvg.rope()), 0, 2, 2, ctypes.c_void_p(1), ctypes.c_void_p(2),
                        None) == -2
