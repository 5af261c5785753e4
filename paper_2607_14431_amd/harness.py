"""Drives the C ABI over the synthetic workloads: the paper's fresh-versus-graft protocol.

Fresh arm: a paged cache is filled by a fresh computation of the prefix (cold prefill),
then the suffix is prefilled and decoding advances token by token on top of it.
Graft arm: the prefix's KV state is deposited as an artifact and grafted into a second
cache (different physical page permutation, different poison in unowned slots); the same
suffix and decode calls then run on it.  Sec. 3.2 (Eq. 1) requires the two arms' outputs
to be byte-identical at the block's own position.

Raw inputs come from the seeded generator (synth.gpu); every computation goes through the
library (paper_2607_14431_amd.kvg).  torch only allocates memory, compares and hashes.
"""

from __future__ import annotations

import dataclasses
import hashlib

import numpy as np
import torch

from synth import ROLE_K, ROLE_Q, ROLE_V
from synth.gpu import raw_chunk
from synth.workloads import Workload

from . import kvg

POISON = {("bf16", 0): 0x7FC1, ("bf16", 1): -0x003D, ("f32", 0): 0x7FC00001, ("f32", 1): -0x003FFFFD,
          ("fp8", 0): 0x7F, ("fp8", 1): 0xFF}
POISON_VIEW = {"bf16": torch.int16, "f32": torch.int32, "fp8": torch.uint8}


def torch_dtype(w: Workload):
    """Storage dtype of the workload's cache."""
    return {"bf16": torch.bfloat16, "f32": torch.float32, "fp8": torch.float8_e4m3fn}[w.dtype]


@dataclasses.dataclass
class Arm:
    w: Workload
    seqs: list
    cache: kvg.Cache
    tables: torch.Tensor        # [B][pages_per_seq] int32 on device
    start_pos: int
    ws: torch.Tensor | None = None
    dws: torch.Tensor | None = None
    shared_tokens: int = 0      # leading tokens whose pages every sequence shares

    @property
    def batch(self):
        return len(self.seqs)

    def meta(self, ctx: int) -> kvg.Seqs:
        B = self.batch
        return kvg.Seqs(self.tables, torch.full((B,), ctx, dtype=torch.int32, device="cuda"),
                        torch.full((B,), self.start_pos, dtype=torch.int64, device="cuda"), ctx,
                        self.shared_tokens)

    def decode_workspace(self, nbytes: int) -> torch.Tensor:
        """Scratch for the decode calls (kept apart from the prefill scratch)."""
        if self.dws is None or self.dws.nbytes < nbytes:
            self.dws = None
            self.dws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
        return self.dws

    def workspace(self, nbytes: int) -> torch.Tensor:
        if self.ws is None or self.ws.nbytes < nbytes:
            self.ws = None
            self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
        return self.ws


def new_arm(w: Workload, seqs, n_ctx: int, seed: int, poison_id: int, start_pos: int | None = None,
            spare_pages: int = 0) -> Arm:
    """A cache holding len(seqs) sequences of up to n_ctx tokens, pages assigned by a
    seeded permutation, every slot filled with a NaN poison pattern."""
    B = len(seqs)
    per_seq = w.pages_for(n_ctx)
    n_pages = B * per_seq + spare_pages
    perm = np.random.default_rng(seed).permutation(n_pages)[: B * per_seq].astype(np.int32)
    tables = torch.from_numpy(perm.reshape(B, per_seq)).cuda()
    cache = kvg.Cache.allocate(w.n_layers, n_pages, w.n_q_heads, w.n_kv_heads, w.head_dim, torch_dtype(w),
                               windows=w.layer_windows)
    bits = POISON[(w.dtype, poison_id)]
    view = POISON_VIEW[w.dtype]
    cache.k_pool.view(view).fill_(bits)
    cache.v_pool.view(view).fill_(bits)
    return Arm(w, list(seqs), cache, tables, w.start_pos if start_pos is None else start_pos)


def rope_of(w: Workload):
    return kvg.rope(w.rope_base, kvg.KVG_ROPE_HALF)


def prefill(arm: Arm, t0: int, n: int, append_only: bool = False, q_sigma_log2=None) -> torch.Tensor | None:
    """Prefill logical tokens [t0, t0 + n) of every sequence of the arm (cache holds [0, t0))."""
    w = arm.w
    k = raw_chunk(w, ROLE_K, arm.seqs, t0, n)
    v = raw_chunk(w, ROLE_V, arm.seqs, t0, n)
    meta = arm.meta(t0)
    if append_only:
        kvg.kvg_append(arm.cache, meta, rope_of(w), 0, w.n_layers, n, k, v)
        return None
    q = raw_chunk(w, ROLE_Q, arm.seqs, t0, n, sigma_log2=q_sigma_log2)
    out = torch.empty((w.n_layers, arm.batch, n, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    ws = arm.workspace(kvg.kvg_prefill_workspace_bytes(arm.cache, meta, w.n_layers, n))
    kvg.kvg_prefill_attn(arm.cache, meta, rope_of(w), 0, w.n_layers, n, q, k, v, w.scale, out, ws)
    return out


def decode(arm: Arm, t0: int, steps: int, q_sigma_log2=None) -> torch.Tensor:
    """Decode steps for logical tokens t0, t0 + 1, ...; returns [steps][L][B][Hq][D] fp32."""
    w = arm.w
    out = torch.empty((steps, w.n_layers, arm.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    for i in range(steps):
        t = t0 + i
        q = raw_chunk(w, ROLE_Q, arm.seqs, t, 1, sigma_log2=q_sigma_log2)
        k = raw_chunk(w, ROLE_K, arm.seqs, t, 1)
        v = raw_chunk(w, ROLE_V, arm.seqs, t, 1)
        meta = arm.meta(t)
        ws = arm.decode_workspace(kvg.kvg_decode_workspace_bytes(arm.cache, meta, w.n_layers))
        kvg.kvg_decode_attn(arm.cache, meta, rope_of(w), 0, w.n_layers, q, k, v, w.scale, out[i], ws)
    return out


def deposit(arm: Arm, bi: int, first: int, n: int, own_pos: int):
    """Deposit tokens [first, first + n) of sequence index bi: (header, payload)."""
    payload = torch.empty(kvg.kvg_payload_bytes(arm.cache, n), dtype=torch.uint8, device="cuda")
    kvg.kvg_deposit(arm.cache, arm.tables[bi], first, n, payload)
    hdr = kvg.kvg_artifact_header_init(arm.cache, n, own_pos, rope_of(arm.w))
    return hdr, payload


def graft(arm: Arm, bi: int, hdr, payload: torch.Tensor, first: int, target_pos: int, relocate: bool = False):
    kvg.kvg_graft(arm.cache, hdr, payload, arm.tables[bi], first, target_pos,
                  kvg.KVG_GRAFT_ALLOW_RELOCATE if relocate else 0)


def sha256_tensor(t: torch.Tensor) -> str:
    """SHA-256 of a tensor's raw bytes (copied to the host in chunks)."""
    h = hashlib.sha256()
    flat = t.contiguous().view(torch.uint8).reshape(-1)
    step = 1 << 28
    for i in range(0, flat.numel(), step):
        h.update(flat[i:i + step].cpu().numpy().tobytes())
    return h.hexdigest()


def bytes_equal(a: torch.Tensor, b: torch.Tensor) -> bool:
    return a.shape == b.shape and torch.equal(a.contiguous().view(torch.uint8), b.contiguous().view(torch.uint8))


@dataclasses.dataclass
class ArmResult:
    suffix: torch.Tensor        # [L][B][S][Hq][D]
    decode: torch.Tensor        # [steps][L][B][Hq][D]

    def digest(self) -> str:
        h = hashlib.sha256()
        for t in (self.suffix, self.decode):
            flat = t.contiguous().view(torch.uint8).reshape(-1)
            step = 1 << 28
            for i in range(0, flat.numel(), step):
                h.update(flat[i:i + step].cpu().numpy().tobytes())
        return h.hexdigest()


def continue_arm(arm: Arm, q_sigma_log2=None) -> ArmResult:
    """Suffix prefill on top of the cached prefix, then decode steps."""
    w = arm.w
    suf = prefill(arm, w.prefix, w.suffix, q_sigma_log2=q_sigma_log2)
    dec = decode(arm, w.prefix + w.suffix, w.decode_steps, q_sigma_log2=q_sigma_log2)
    return ArmResult(suf, dec)


def fresh_prefix(arm: Arm, append_only: bool = False, chunk: int | None = None):
    """Cold computation of the prefix [0, w.prefix), in chunks of `chunk` tokens."""
    w = arm.w
    chunk = w.prefix if chunk is None else chunk
    for t0 in range(0, w.prefix, chunk):
        prefill(arm, t0, min(chunk, w.prefix - t0), append_only=append_only)


def store_artifact(w: Workload, block: int, slot: int, seed: int = 991):
    """Artifact of store block `block` captured at its own position slot * block_tokens:
    a fresh computation of the block in a scratch cache, then a deposit."""
    from synth.workloads import STORE_UNIT
    n = w.store_block_tokens(block)
    own = slot * w.block_tokens
    sw = dataclasses.replace(w, blocks_per_seq=1, block_tokens=0, prefix=n, suffix=0, decode_steps=0,
                             batch=1, fixed_unit=STORE_UNIT + block)
    scratch = new_arm(sw, [0], n, seed, 0, start_pos=own)
    prefill(scratch, 0, n, append_only=True)
    return deposit(scratch, 0, 0, n, own)


# ----------------------------------------------------------------------------------------
# Large-store paging (Sec. 4.4): a serving window of `slots` direct-mapped block slots,
# shared by `batch` sequences, each with private suffix pages.  Block b of the store lives
# in host-pinned memory and is grafted into slot b mod slots, its own position; the graft
# kernel reads the pinned payload over PCIe.

_hip = None


def _hip_runtime():
    global _hip
    if _hip is None:
        import ctypes
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipHostGetDevicePointer.restype = ctypes.c_int
        _hip.hipHostGetDevicePointer.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_uint]
    return _hip


class PinnedPayload:
    """A host-pinned payload buffer and the device address through which kernels read it."""

    def __init__(self, nbytes: int):
        import ctypes
        self.host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
        dev = ctypes.c_void_p()
        rc = _hip_runtime().hipHostGetDevicePointer(ctypes.byref(dev), ctypes.c_void_p(self.host.data_ptr()), 0)
        if rc != 0 or not dev.value:
            raise RuntimeError(f"pinned payload is not device-accessible (hipHostGetDevicePointer rc={rc})")
        self.dev_ptr = dev.value
        self.nbytes = nbytes

    def data_ptr(self):                      # what kvg_graft receives
        return self.dev_ptr


def artifact_workspace(hdr) -> torch.Tensor:
    """Device scratch for kvg_artifact_seal / kvg_artifact_verify of this header's payload."""
    return torch.empty(max(kvg.kvg_artifact_digest_workspace_bytes(hdr), 256), dtype=torch.uint8, device="cuda")


def save_artifact(path: str, hdr, payload: torch.Tensor):
    """The block's file form: the header's bytes, then the payload's (device tensor, copied to
    the host in chunks)."""
    import ctypes
    flat = payload.contiguous().view(torch.uint8).reshape(-1)[: hdr.payload_bytes]
    with open(path, "wb") as f:
        f.write(ctypes.string_at(ctypes.addressof(hdr), ctypes.sizeof(hdr)))
        step = 1 << 28
        for i in range(0, flat.numel(), step):
            f.write(flat[i:i + step].cpu().numpy().tobytes())


def load_artifact(path: str):
    """Read a block's file into (header, PinnedPayload): the payload lands in host-pinned memory,
    from which kvg_artifact_verify and kvg_graft read it over PCIe."""
    import ctypes
    import os
    size = os.path.getsize(path)
    hsize = ctypes.sizeof(kvg.kvg_artifact_hdr)
    with open(path, "rb") as f:
        hdr = kvg.kvg_artifact_hdr.from_buffer_copy(f.read(hsize))
        if size != hsize + hdr.payload_bytes:
            raise ValueError(f"{path}: {size} bytes, header says {hsize} + {hdr.payload_bytes}")
        pinned = PinnedPayload(hdr.payload_bytes)
        view = memoryview(pinned.host.numpy())
        got = 0
        while got < hdr.payload_bytes:
            n = f.readinto(view[got:])
            if not n:
                raise ValueError(f"{path}: short read")
            got += n
    return hdr, pinned


class StoreWindow:
    """The serving window: `slots` direct-mapped block slots shared by every sequence (the
    leading block-table entries of all rows are the same pages), then each sequence's private
    pages for its suffix and decode tokens.  Pages are laid out in order, or (permute_seed)
    by a seeded permutation; unwritten slots hold the NaN poison of `poison_id`."""

    def __init__(self, w: Workload, batch: int | None = None, permute_seed: int | None = None, poison_id: int = 1,
                 extra_tokens: int = 0):
        from synth.workloads import STORE_UNIT
        self.w = w
        self.batch = w.batch if batch is None else batch
        self.slots = w.blocks_per_seq
        self.slot_pages = w.block_tokens // w.page_size
        self.win_tokens = self.slots * w.block_tokens
        tail = w.suffix + w.decode_steps + extra_tokens
        self.suf_pages = w.pages_for(tail)
        n_win = self.slots * self.slot_pages
        n_pages = n_win + self.batch * self.suf_pages
        order = (np.arange(n_pages) if permute_seed is None
                 else np.random.default_rng(permute_seed).permutation(n_pages)).astype(np.int32)
        rows = []
        for s in range(self.batch):
            own = order[n_win + s * self.suf_pages: n_win + (s + 1) * self.suf_pages]
            rows.append(np.concatenate([order[:n_win], own]))
        self.tables = torch.from_numpy(np.stack(rows)).cuda()
        self.cache = kvg.Cache.allocate(w.n_layers, n_pages, w.n_q_heads, w.n_kv_heads, w.head_dim, torch_dtype(w),
                               windows=w.layer_windows)
        view = POISON_VIEW[w.dtype]
        self.cache.k_pool.view(view).fill_(POISON[(w.dtype, poison_id)])
        self.cache.v_pool.view(view).fill_(POISON[(w.dtype, poison_id)])
        self.history = [[] for _ in range(self.slots)]   # (block, n_tokens) grafted into each slot
        self.unit0 = STORE_UNIT
        self.arm = Arm(dataclasses.replace(w, prefix=self.win_tokens, batch=self.batch), list(range(self.batch)),
                       self.cache, self.tables, 0, shared_tokens=self.win_tokens)

    def materialize(self, b: int, pinned: PinnedPayload):
        """Deposit of store block b (fresh computation at its own position, then the gather)
        copied into host-pinned memory: the store's on-host form of the block."""
        hdr, payload = store_artifact(self.w, b, b % self.slots)
        pinned.host[: payload.numel()].copy_(payload)
        torch.cuda.synchronize()
        return hdr

    def graft(self, b: int, hdr, pinned: PinnedPayload, stream=None):
        """Restore block b from host-pinned memory into slot b mod slots (shared pages)."""
        j = b % self.slots
        first = j * self.w.block_tokens
        kvg._check(kvg._lib.kvg_graft(kvg.ctypes.byref(self.cache.struct()), kvg.ctypes.byref(hdr),
                                      kvg.ctypes.c_void_p(pinned.data_ptr()), kvg._ptr(self.tables[0]),
                                      self.tables.shape[1], first, first, 0, kvg._stream(stream)), "kvg_graft")
        self.history[j].append((b, self.w.store_block_tokens(b)))

    def append_block(self, b: int):
        """Fresh computation of store block b into slot b mod slots at its own position: the
        block's raw keys rotated and stored, its values copied, through the shared pages."""
        from synth.workloads import STORE_UNIT
        j = b % self.slots
        n = self.w.store_block_tokens(b)
        sw = dataclasses.replace(self.w, blocks_per_seq=1, block_tokens=0, prefix=n, suffix=0, decode_steps=0,
                                 batch=1, fixed_unit=STORE_UNIT + b)
        k = raw_chunk(sw, ROLE_K, [0], 0, n)
        v = raw_chunk(sw, ROLE_V, [0], 0, n)
        first = j * self.w.block_tokens
        meta = kvg.Seqs(self.tables[:1].contiguous(), torch.full((1,), first, dtype=torch.int32, device="cuda"),
                        torch.zeros(1, dtype=torch.int64, device="cuda"), first)
        kvg.kvg_append(self.cache, meta, rope_of(self.w), 0, self.w.n_layers, n, k, v)
        self.history[j].append((b, n))

    def segments(self):
        """Generator runs describing the window's contents (for the oracle and the inputs)."""
        segs = []
        for j in range(self.slots):
            base = j * self.w.block_tokens
            filled = 0
            runs = []
            for (b, n) in reversed(self.history[j]):        # newest first
                if n > filled:
                    runs.append((base + filled, n - filled, self.unit0 + b, filled))
                    filled = n
                if filled >= self.w.block_tokens:
                    break
            if filled < self.w.block_tokens:
                raise RuntimeError(f"slot {j} is not fully written")
            segs.extend(sorted(runs))
        return tuple(segs)

    def view(self) -> Workload:
        """The workload as the sequences see it now: window contents, then their own tokens."""
        return dataclasses.replace(self.w, prefix=self.win_tokens, batch=self.batch,
                                   explicit_segments=self.segments(), blocks_per_seq=1, block_tokens=0)


# ----------------------------------------------------------------------------------------
# Logit-level verdict (Eq. 1-2, Sec. 4.1's table): a synthetic soft-capped head over the last
# layer's attention outputs (heads concatenated), SHA-256 of every logit row, the KL
# divergence and argmax of graft against fresh, and the Mann-Whitney U test of those KLs
# against a noise floor (fresh against a second fresh run) with Cliff's delta.

HEAD_VOCAB = 262_144      # vocabulary of the 12B-class model family
HEAD_CAP = 30.0           # final-logit soft cap of that family
HEAD_SIGMA_LOG2 = 3       # weight scale: attention outputs average many value rows (|o| ~ 0.02
                          # at the 12B-class shapes), so sigma 8 puts the largest logits at the cap


@dataclasses.dataclass
class Head:
    packed: torch.Tensor        # weights as kvg_logits_pack leaves them
    vocab: int
    hidden: int


def head_weights(w: Workload, vocab: int = HEAD_VOCAB, sigma_log2: int = HEAD_SIGMA_LOG2) -> Head:
    """Seeded bf16 weights [vocab][Hq * D] of the synthetic head, packed on the device."""
    from synth import ROLE_W
    from synth.gpu import fill
    H = w.n_q_heads * w.head_dim
    rowmajor = torch.empty((vocab, H), dtype=torch.bfloat16, device="cuda")
    fill(rowmajor, 0, 1, 0, 0, vocab, 1, H, w.seed, w.stream(ROLE_W, 0).id, sigma_log2, True)
    return pack_head(rowmajor)


def pack_head(rowmajor: torch.Tensor) -> Head:
    vocab, H = rowmajor.shape
    packed = torch.empty(kvg.kvg_logits_packed_bytes(vocab, H), dtype=torch.uint8, device="cuda")
    kvg.kvg_logits_pack(rowmajor, packed)
    return Head(packed, vocab, H)


def hidden_rows(res: ArmResult, bi: int, rows=None) -> torch.Tensor:
    """Last layer's outputs of sequence index bi for its suffix rows then its decode steps,
    heads concatenated: fp32 [n][Hq * D]; `rows` selects among them."""
    suf = res.suffix[-1, bi]                              # [S][Hq][D]
    dec = res.decode[:, -1, bi]                           # [steps][Hq][D]
    allr = torch.cat([suf, dec], dim=0)
    allr = allr.reshape(allr.shape[0], -1)
    return (allr if rows is None else allr[list(rows)]).contiguous()


def logits(hidden: torch.Tensor, head: Head, cap: float = HEAD_CAP) -> torch.Tensor:
    rows = hidden.shape[0]
    out = torch.empty((rows, head.vocab), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(kvg.kvg_logits_workspace_bytes(rows, hidden.shape[1]), 256), dtype=torch.uint8,
                     device="cuda")
    kvg.kvg_logits(hidden, head.packed, head.vocab, cap, out, ws)
    return out


def row_digests(x: torch.Tensor) -> torch.Tensor:
    """SHA-256 of each row's bytes (uint8 [rows][32], device)."""
    rows = x.shape[0]
    row_bytes = x[0].numel() * x.element_size()
    dig = torch.empty((rows, 32), dtype=torch.uint8, device="cuda")
    kvg.kvg_leaf_digests(x, row_bytes, dig)
    return dig


def compare_logits(a: torch.Tensor, b: torch.Tensor):
    """Per row: KL(softmax(a) || softmax(b)) (fp64), argmax of a, argmax of b (host arrays)."""
    rows = a.shape[0]
    kl = torch.empty(rows, dtype=torch.float64, device="cuda")
    ia = torch.empty(rows, dtype=torch.int32, device="cuda")
    ib = torch.empty(rows, dtype=torch.int32, device="cuda")
    kvg.kvg_logit_compare(a, b, kl, ia, ib)
    return kl.cpu().numpy(), ia.cpu().numpy(), ib.cpu().numpy()


def exactness_stats(graft: torch.Tensor, fresh: torch.Tensor, noise: torch.Tensor | None = None) -> dict:
    """The paper's per-sample verdict over logit rows (each row one sample): byte equality
    by SHA-256, KL median / p99, argmax disagreements, and against the noise floor (fresh
    against `noise`, a second fresh run) the two-sided Mann-Whitney p and Cliff's delta."""
    import scipy.stats
    n = graft.shape[0]
    same = (row_digests(graft) == row_digests(fresh)).all(dim=1).cpu().numpy()
    kl, ia, ib = compare_logits(graft, fresh)
    out = {"samples": n, "sha256_equal": int(same.sum()), "kl_median": float(np.median(kl)),
           "kl_p99": float(np.percentile(kl, 99)), "argmax_disagree": int((ia != ib).sum())}
    if noise is not None:
        floor, _, _ = compare_logits(noise, fresh)
        if np.all(kl == kl[0]) and np.all(floor == kl[0]):
            p = 1.0                     # every value tied: no evidence of a difference
        else:
            p = float(scipy.stats.mannwhitneyu(kl, floor, alternative="two-sided", method="asymptotic").pvalue)
        gt = (kl[:, None] > floor[None, :]).sum()
        lt = (kl[:, None] < floor[None, :]).sum()
        out.update({"noise_kl_median": float(np.median(floor)), "mann_whitney_p": p,
                    "cliffs_delta": float((gt - lt) / (n * len(floor)))})
    return out
