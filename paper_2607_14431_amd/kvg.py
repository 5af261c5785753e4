"""Python binding of libkvg.so: same names as the C ABI (include/kvg.h), argument
marshalling only.  Every step runs in the library's HIP kernels; torch supplies device
memory and the stream.  Importing this module without the built library raises.
"""

from __future__ import annotations

import ctypes
import dataclasses
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvg.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_14431_amd.build` "
                      "(there is no fallback path)")
_lib = ctypes.CDLL(LIB_PATH)

KVG_F32, KVG_BF16, KVG_FP8_E4M3 = 0, 1, 2
KVG_ROPE_HALF, KVG_ROPE_INTERLEAVED = 0, 1
KVG_GRAFT_ALLOW_RELOCATE = 1
KVG_ARTIFACT_MAGIC = 0x4147564B
KVG_ARTIFACT_VERSION = 2

STATUS = {
    0: "KVG_OK", -1: "KVG_E_INVAL", -2: "KVG_E_SHAPE", -3: "KVG_E_DTYPE", -4: "KVG_E_POSITION",
    -5: "KVG_E_CAPACITY", -6: "KVG_E_ALIGN", -7: "KVG_E_CORRUPT", -8: "KVG_E_HIP", -9: "KVG_E_WORKSPACE",
}


class KvgError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        self.name = STATUS.get(status, str(status))
        super().__init__(f"{where}: {self.name} ({kvg_status_str(status)})")


class kvg_rope(ctypes.Structure):
    _fields_ = [("base", ctypes.c_double), ("pairing", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class kvg_cache(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("n_pages", ctypes.c_int64), ("k_pool", ctypes.c_void_p), ("v_pool", ctypes.c_void_p),
                ("layer_window", ctypes.POINTER(ctypes.c_int32))]


class kvg_seqs(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("max_pages", ctypes.c_int32), ("max_ctx_len", ctypes.c_int32),
                ("shared_tokens", ctypes.c_int32), ("block_tables", ctypes.c_void_p), ("ctx_lens", ctypes.c_void_p),
                ("start_pos", ctypes.c_void_p)]


class kvg_artifact_hdr(ctypes.Structure):
    _fields_ = [("magic", ctypes.c_uint32), ("version", ctypes.c_uint32), ("dtype", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("n_tokens", ctypes.c_int32), ("own_pos", ctypes.c_int64),
                ("rope_base", ctypes.c_double), ("rope_pairing", ctypes.c_int32),
                ("digest_leaf_bytes", ctypes.c_uint32), ("payload_bytes", ctypes.c_uint64),
                ("digest", ctypes.c_uint8 * 32)]


_P = ctypes.POINTER
_vp, _i32, _i64, _sz, _f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
_u64 = ctypes.c_uint64

_SIGS = {
    "kvg_version": (ctypes.c_char_p, []),
    "kvg_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "kvg_payload_bytes": (_sz, [_P(kvg_cache), _i32]),
    "kvg_artifact_header_init": (ctypes.c_int, [_P(kvg_cache), _i32, _i64, _P(kvg_rope), _P(kvg_artifact_hdr)]),
    "kvg_artifact_digest_workspace_bytes": (_sz, [_P(kvg_artifact_hdr)]),
    "kvg_artifact_seal": (ctypes.c_int, [_P(kvg_artifact_hdr), _vp, _vp, _sz, _vp]),
    "kvg_artifact_verify": (ctypes.c_int, [_P(kvg_artifact_hdr), _vp, _vp, _sz, _vp]),
    "kvg_append": (ctypes.c_int, [_P(kvg_cache), _P(kvg_seqs), _P(kvg_rope), _i32, _i32, _i32, _vp, _vp, _vp]),
    "kvg_deposit": (ctypes.c_int, [_P(kvg_cache), _vp, _i32, _i32, _i32, _vp, _vp]),
    "kvg_graft": (ctypes.c_int, [_P(kvg_cache), _P(kvg_artifact_hdr), _vp, _vp, _i32, _i32, _i64, _i32, _vp]),
    "kvg_prefill_workspace_bytes": (_sz, [_P(kvg_cache), _P(kvg_seqs), _i32, _i32]),
    "kvg_prefill_attn": (ctypes.c_int, [_P(kvg_cache), _P(kvg_seqs), _P(kvg_rope), _i32, _i32, _i32, _vp, _vp,
                                        _vp, _f32, _vp, _vp, _sz, _vp]),
    "kvg_decode_workspace_bytes": (_sz, [_P(kvg_cache), _P(kvg_seqs), _i32]),
    "kvg_decode_attn": (ctypes.c_int, [_P(kvg_cache), _P(kvg_seqs), _P(kvg_rope), _i32, _i32, _vp, _vp, _vp,
                                       _f32, _vp, _vp, _sz, _vp]),
    "kvg_decode_attn_noalloc": (ctypes.c_int, [_P(kvg_cache), _P(kvg_seqs), _P(kvg_rope), _i32, _i32, _vp, _vp, _vp,
                                               _f32, _vp, _vp]),
    "kvg_leaf_digests": (ctypes.c_int, [_vp, _u64, ctypes.c_uint32, _vp, _vp]),
    "kvg_merkle_workspace_bytes": (_sz, [_u64]),
    "kvg_merkle_root": (ctypes.c_int, [_vp, _u64, _vp, _vp, _sz, _vp]),
    "kvg_dedup_workspace_bytes": (_sz, [_u64]),
    "kvg_dedup_map": (ctypes.c_int, [_vp, _u64, _vp, _vp, _vp, _sz, _vp]),
    "kvg_logits_packed_bytes": (_sz, [_i32, _i32]),
    "kvg_logits_pack": (ctypes.c_int, [_vp, _i32, _i32, _vp, _vp]),
    "kvg_logits_workspace_bytes": (_sz, [_i32, _i32]),
    "kvg_logits": (ctypes.c_int, [_vp, _i32, _i32, _vp, _i32, _f32, _vp, _vp, _sz, _vp]),
    "kvg_logit_compare": (ctypes.c_int, [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTED = tuple(_SIGS)


def kvg_version() -> str:
    return _lib.kvg_version().decode()


def kvg_status_str(status: int) -> str:
    return _lib.kvg_status_str(status).decode()


def _check(status: int, where: str):
    if status != 0:
        raise KvgError(status, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def rope(base: float = 10000.0, pairing: int = KVG_ROPE_HALF) -> kvg_rope:
    return kvg_rope(base, pairing, 0)


@dataclasses.dataclass
class Cache:
    """Paged pools [n_layers][n_pages][n_kv_heads][page_size][head_dim] (torch tensors)."""
    k_pool: torch.Tensor
    v_pool: torch.Tensor
    n_q_heads: int
    windows: tuple | None = None       # per-layer sliding window (0 = full causal), or None

    @staticmethod
    def allocate(n_layers, n_pages, n_q_heads, n_kv_heads, head_dim, dtype: torch.dtype, device="cuda",
                 page_size=16, windows=None):
        shape = (n_layers, n_pages, n_kv_heads, page_size, head_dim)
        if windows is not None:
            windows = tuple(int(x) for x in windows)
            assert len(windows) == n_layers
        return Cache(torch.empty(shape, dtype=dtype, device=device),
                     torch.empty(shape, dtype=dtype, device=device), n_q_heads, windows)

    @property
    def n_layers(self):
        return self.k_pool.shape[0]

    @property
    def n_pages(self):
        return self.k_pool.shape[1]

    @property
    def n_kv_heads(self):
        return self.k_pool.shape[2]

    @property
    def page_size(self):
        return self.k_pool.shape[3]

    @property
    def head_dim(self):
        return self.k_pool.shape[4]

    @property
    def kvg_dtype(self):
        return {torch.float32: KVG_F32, torch.bfloat16: KVG_BF16,
                torch.float8_e4m3fn: KVG_FP8_E4M3}[self.k_pool.dtype]

    @property
    def raw_dtype(self) -> torch.dtype:
        """dtype of the raw q/k/v this cache takes (bf16 for an fp8 cache)."""
        return torch.bfloat16 if self.k_pool.dtype == torch.float8_e4m3fn else self.k_pool.dtype

    def struct(self) -> kvg_cache:
        assert self.k_pool.is_contiguous() and self.v_pool.is_contiguous()
        assert self.k_pool.shape == self.v_pool.shape and self.k_pool.dtype == self.v_pool.dtype
        c = kvg_cache(self.n_layers, self.n_q_heads, self.n_kv_heads, self.head_dim, self.page_size,
                      self.kvg_dtype, self.n_pages, self.k_pool.data_ptr(), self.v_pool.data_ptr(), None)
        if self.windows is not None and any(self.windows):
            arr = (ctypes.c_int32 * len(self.windows))(*self.windows)
            c.layer_window = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32))
            c._windows_keepalive = arr        # the struct holds a raw pointer into this array
        return c


@dataclasses.dataclass
class Seqs:
    """Block tables [batch][max_pages] int32, ctx_lens [batch] int32, start_pos [batch] int64 (device);
    shared_tokens: leading tokens whose table entries all sequences share (0 = none)."""
    block_tables: torch.Tensor
    ctx_lens: torch.Tensor
    start_pos: torch.Tensor
    max_ctx_len: int
    shared_tokens: int = 0      # leading tokens every sequence's table shares (see kvg_seqs in kvg.h)

    def struct(self) -> kvg_seqs:
        bt = self.block_tables
        assert bt.dtype == torch.int32 and bt.is_contiguous() and bt.dim() == 2
        assert self.ctx_lens.dtype == torch.int32 and self.start_pos.dtype == torch.int64
        return kvg_seqs(bt.shape[0], bt.shape[1], self.max_ctx_len, self.shared_tokens, bt.data_ptr(),
                        self.ctx_lens.data_ptr(), self.start_pos.data_ptr())


def kvg_payload_bytes(cache: Cache, n_tokens: int) -> int:
    return _lib.kvg_payload_bytes(ctypes.byref(cache.struct()), n_tokens)


def kvg_artifact_header_init(cache: Cache, n_tokens: int, own_pos: int, rp: kvg_rope) -> kvg_artifact_hdr:
    hdr = kvg_artifact_hdr()
    _check(_lib.kvg_artifact_header_init(ctypes.byref(cache.struct()), n_tokens, own_pos, ctypes.byref(rp),
                                         ctypes.byref(hdr)), "kvg_artifact_header_init")
    return hdr


def kvg_artifact_digest_workspace_bytes(hdr: kvg_artifact_hdr) -> int:
    return _lib.kvg_artifact_digest_workspace_bytes(ctypes.byref(hdr))


def _payload_ptr(payload):
    """Device address of a payload: a torch tensor, or an object with data_ptr() (pinned host
    memory exposed through its device address)."""
    return ctypes.c_void_p(payload.data_ptr())


def kvg_artifact_seal(hdr: kvg_artifact_hdr, payload, ws: torch.Tensor, stream=None):
    _check(_lib.kvg_artifact_seal(ctypes.byref(hdr), _payload_ptr(payload), _ptr(ws), ws.nbytes, _stream(stream)),
           "kvg_artifact_seal")


def kvg_artifact_verify(hdr: kvg_artifact_hdr, payload, ws: torch.Tensor, stream=None) -> int:
    """Status of the verification: 0 (KVG_OK) or KVG_E_CORRUPT (-7); other errors raise."""
    st = _lib.kvg_artifact_verify(ctypes.byref(hdr), _payload_ptr(payload), _ptr(ws), ws.nbytes, _stream(stream))
    if st not in (0, -7):
        raise KvgError(st, "kvg_artifact_verify")
    return st


def _raw_ok(cache: Cache, *raws):
    for t in raws:
        assert t.dtype == cache.raw_dtype and t.is_contiguous(), "raw inputs: the cache's raw dtype, contiguous"


def kvg_append(cache: Cache, seqs: Seqs, rp: kvg_rope, layer0: int, n_layers: int, chunk_len: int,
               k_raw: torch.Tensor, v_raw: torch.Tensor, stream=None):
    _raw_ok(cache, k_raw, v_raw)
    _check(_lib.kvg_append(ctypes.byref(cache.struct()), ctypes.byref(seqs.struct()), ctypes.byref(rp), layer0,
                           n_layers, chunk_len, _ptr(k_raw), _ptr(v_raw), _stream(stream)), "kvg_append")


def kvg_deposit(cache: Cache, block_table_row: torch.Tensor, first_token: int, n_tokens: int,
                payload: torch.Tensor, stream=None):
    assert payload.nbytes >= kvg_payload_bytes(cache, n_tokens)
    _check(_lib.kvg_deposit(ctypes.byref(cache.struct()), _ptr(block_table_row), block_table_row.numel(),
                            first_token, n_tokens, _ptr(payload), _stream(stream)), "kvg_deposit")


def kvg_graft(cache: Cache, hdr: kvg_artifact_hdr, payload: torch.Tensor, block_table_row: torch.Tensor,
              first_token: int, target_pos: int, flags: int = 0, stream=None):
    assert payload.nbytes >= hdr.payload_bytes
    _check(_lib.kvg_graft(ctypes.byref(cache.struct()), ctypes.byref(hdr), _ptr(payload), _ptr(block_table_row),
                          block_table_row.numel(), first_token, target_pos, flags, _stream(stream)), "kvg_graft")


def kvg_prefill_workspace_bytes(cache: Cache, seqs: Seqs, n_layers: int, chunk_len: int) -> int:
    return _lib.kvg_prefill_workspace_bytes(ctypes.byref(cache.struct()), ctypes.byref(seqs.struct()), n_layers,
                                            chunk_len)


def kvg_prefill_attn(cache: Cache, seqs: Seqs, rp: kvg_rope, layer0: int, n_layers: int, chunk_len: int,
                     q_raw, k_raw, v_raw, scale: float, out: torch.Tensor, ws: torch.Tensor, stream=None):
    _raw_ok(cache, q_raw, k_raw, v_raw)
    _check(_lib.kvg_prefill_attn(ctypes.byref(cache.struct()), ctypes.byref(seqs.struct()), ctypes.byref(rp),
                                 layer0, n_layers, chunk_len, _ptr(q_raw), _ptr(k_raw), _ptr(v_raw), scale,
                                 _ptr(out), _ptr(ws), ws.nbytes, _stream(stream)), "kvg_prefill_attn")


def kvg_decode_workspace_bytes(cache: Cache, seqs: Seqs, n_layers: int) -> int:
    return _lib.kvg_decode_workspace_bytes(ctypes.byref(cache.struct()), ctypes.byref(seqs.struct()), n_layers)


def decode_workspace(cache: Cache, seqs: Seqs, n_layers: int) -> torch.Tensor:
    """Scratch for kvg_decode_attn sized for `seqs` (covers any call with max_ctx_len no larger)."""
    return torch.empty(max(kvg_decode_workspace_bytes(cache, seqs, n_layers), 256), dtype=torch.uint8,
                       device=cache.k_pool.device)


def kvg_decode_attn(cache: Cache, seqs: Seqs, rp: kvg_rope, layer0: int, n_layers: int, q_raw, k_raw, v_raw,
                    scale: float, out: torch.Tensor, ws: torch.Tensor, stream=None):
    _raw_ok(cache, q_raw, k_raw, v_raw)
    _check(_lib.kvg_decode_attn(ctypes.byref(cache.struct()), ctypes.byref(seqs.struct()), ctypes.byref(rp),
                                layer0, n_layers, _ptr(q_raw), _ptr(k_raw), _ptr(v_raw), scale, _ptr(out), _ptr(ws),
                                ws.nbytes, _stream(stream)), "kvg_decode_attn")


KVG_NOALLOC_SCRATCH_BYTES = 256 << 20


def kvg_decode_attn_noalloc(cache: Cache, seqs: Seqs, rp: kvg_rope, layer0: int, n_layers: int, q_raw, k_raw, v_raw,
                            scale: float, out: torch.Tensor, stream=None):
    """kvg_decode_attn on the library's own fixed workspace (no allocation by anyone)."""
    _raw_ok(cache, q_raw, k_raw, v_raw)
    _check(_lib.kvg_decode_attn_noalloc(ctypes.byref(cache.struct()), ctypes.byref(seqs.struct()), ctypes.byref(rp),
                                        layer0, n_layers, _ptr(q_raw), _ptr(k_raw), _ptr(v_raw), scale, _ptr(out),
                                        _stream(stream)), "kvg_decode_attn_noalloc")


def kvg_leaf_digests(data: torch.Tensor, leaf_bytes: int, digests: torch.Tensor, n_bytes: int | None = None,
                     stream=None):
    """SHA-256 of each leaf of `data`'s bytes into `digests` (uint8 [n_leaves][32], device)."""
    nb = data.nbytes if n_bytes is None else n_bytes
    _check(_lib.kvg_leaf_digests(_ptr(data), nb, leaf_bytes, _ptr(digests), _stream(stream)), "kvg_leaf_digests")


def kvg_merkle_workspace_bytes(n_leaves: int) -> int:
    return _lib.kvg_merkle_workspace_bytes(n_leaves)


def kvg_merkle_root(digests: torch.Tensor, n_leaves: int, root: torch.Tensor, ws: torch.Tensor, stream=None):
    _check(_lib.kvg_merkle_root(_ptr(digests), n_leaves, _ptr(root), _ptr(ws), ws.nbytes, _stream(stream)),
           "kvg_merkle_root")


def kvg_dedup_workspace_bytes(n_leaves: int) -> int:
    return _lib.kvg_dedup_workspace_bytes(n_leaves)


def kvg_dedup_map(digests: torch.Tensor, n_leaves: int, first_index: torch.Tensor, n_unresolved: torch.Tensor,
                  ws: torch.Tensor, stream=None):
    _check(_lib.kvg_dedup_map(_ptr(digests), n_leaves, _ptr(first_index), _ptr(n_unresolved), _ptr(ws), ws.nbytes,
                              _stream(stream)), "kvg_dedup_map")


def kvg_logits_packed_bytes(vocab: int, hidden: int) -> int:
    return _lib.kvg_logits_packed_bytes(vocab, hidden)


def kvg_logits_pack(w: torch.Tensor, packed: torch.Tensor, stream=None):
    """w: bf16 [V][H] row-major; packed: kvg_logits_packed_bytes(V, H) bytes (device)."""
    V, H = w.shape
    assert w.dtype == torch.bfloat16 and w.is_contiguous()
    assert packed.nbytes >= kvg_logits_packed_bytes(V, H)
    _check(_lib.kvg_logits_pack(_ptr(w), V, H, _ptr(packed), _stream(stream)), "kvg_logits_pack")


def kvg_logits_workspace_bytes(rows: int, hidden: int) -> int:
    return _lib.kvg_logits_workspace_bytes(rows, hidden)


def kvg_logits(hidden: torch.Tensor, w_packed: torch.Tensor, vocab: int, cap: float, out: torch.Tensor,
               ws: torch.Tensor, stream=None):
    """hidden: fp32 [rows][H]; w_packed: as kvg_logits_pack left it; out: fp32 [rows][vocab]."""
    rows, H = hidden.shape
    assert tuple(out.shape) == (rows, vocab) and w_packed.nbytes >= kvg_logits_packed_bytes(vocab, H)
    assert hidden.dtype == torch.float32 and out.dtype == torch.float32
    assert hidden.is_contiguous() and w_packed.is_contiguous() and out.is_contiguous()
    _check(_lib.kvg_logits(_ptr(hidden), rows, H, _ptr(w_packed), vocab, cap, _ptr(out), _ptr(ws), ws.nbytes,
                           _stream(stream)), "kvg_logits")


def kvg_logit_compare(a: torch.Tensor, b: torch.Tensor, kl: torch.Tensor, argmax_a: torch.Tensor,
                      argmax_b: torch.Tensor, stream=None):
    """a, b: fp32 [rows][V]; kl: fp64 [rows]; argmax_a, argmax_b: int32 [rows] (all device)."""
    rows, V = a.shape
    assert tuple(b.shape) == (rows, V) and a.dtype == b.dtype == torch.float32
    assert a.is_contiguous() and b.is_contiguous()
    assert kl.dtype == torch.float64 and argmax_a.dtype == argmax_b.dtype == torch.int32
    assert kl.numel() >= rows and argmax_a.numel() >= rows and argmax_b.numel() >= rows
    _check(_lib.kvg_logit_compare(_ptr(a), _ptr(b), rows, V, _ptr(kl), _ptr(argmax_a), _ptr(argmax_b),
                                  _stream(stream)), "kvg_logit_compare")


def raw_call(name: str, *args):
    """Direct call of an exported symbol with pre-marshalled ctypes arguments (for validation tests)."""
    return getattr(_lib, name)(*args)
