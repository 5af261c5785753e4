"""The five synthetic workloads: shapes, dtypes, sigmas, seeds and how each
sequence's logical tokens map to generator streams.  Plain data; no method
arithmetic.

Shapes follow the paper's model classes: a 12B-class GQA stack (48 layers, 16
query / 8 KV heads, head_dim 256) and a 31B-class stack (60 layers, 32 / 16,
head_dim 128); the 2,854,766-token store and 32,768-token serving window are
the figures of the paper's long-store experiment (Sec. 4.4).
"""

from __future__ import annotations

import dataclasses

import numpy as np

from .philox import ROLE_K, ROLE_NK, ROLE_NV, ROLE_Q, ROLE_V, Stream

BASE_SEED = 14431
STORE_UNIT = 1 << 20        # stream unit offset for store blocks (unit = STORE_UNIT + block id)


@dataclasses.dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str                 # "f32" | "bf16"
    page_size: int
    prefix: int                # grafted block length (tokens) per sequence
    suffix: int                # suffix prefill chunk
    decode_steps: int
    batch: int
    sigma_log2: int            # K/V (and Q) standard deviation = 2**sigma_log2
    rope_base: float = 10000.0
    start_pos: int = 0         # absolute position of logical token 0 (graft target)
    own_pos: int = 0           # position the block was captured at
    blocks_per_seq: int = 1    # >1: the prefix is several store blocks
    block_tokens: int = 0      # tokens per store block (0: prefix is one private block)
    store_blocks: int = 0      # number of blocks in the seeded store
    store_tokens: int = 0      # total store tokens (last block may be partial)
    seed: int = BASE_SEED
    fixed_unit: int = -1       # >= 0: every sequence draws all tokens from this stream unit
    explicit_segments: tuple = ()   # (t0, n, unit, offset) runs covering [0, prefix), e.g. a window's contents
    sliding_window: int = 0    # > 0: windowed layers attend to the last `sliding_window` keys
    global_every: int = 0      # > 0: every global_every-th layer (1-based) stays global
    needle_span: int = 0       # > 0: every store block carries a needle row at a seeded offset
                               # in [0, needle_span) (at most the shortest block's tokens)

    def layer_window(self, layer: int) -> int:
        """Attention window of a layer: 0 = full causal."""
        if self.sliding_window <= 0:
            return 0
        if self.global_every > 0 and (layer + 1) % self.global_every == 0:
            return 0
        return self.sliding_window

    @property
    def layer_windows(self) -> tuple:
        return tuple(self.layer_window(i) for i in range(self.n_layers))

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def ctx_final(self) -> int:
        return self.prefix + self.suffix + self.decode_steps

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.head_dim))

    @property
    def elem_bytes(self) -> int:
        return {"bf16": 2, "f32": 4, "fp8": 1}[self.dtype]

    @property
    def raw_dtype(self) -> str:
        """dtype of the raw q/k/v the model hands over: an fp8 cache stores bf16 inputs."""
        return "bf16" if self.dtype == "fp8" else self.dtype

    @property
    def page_bytes(self) -> int:
        """One page of one layer, K or V."""
        return self.n_kv_heads * self.page_size * self.head_dim * self.elem_bytes

    def pages_for(self, n_tokens: int) -> int:
        return -(-n_tokens // self.page_size)

    def stream(self, role: int, unit: int) -> Stream:
        return Stream(self.wid, role, unit)

    def store_block_tokens(self, b: int) -> int:
        if not self.store_blocks:
            return self.prefix
        if b < self.store_blocks - 1:
            return self.block_tokens
        return self.store_tokens - self.block_tokens * (self.store_blocks - 1)

    def needle_offset(self, b: int) -> int:
        """Token of store block b whose key and value rows are the block's needle: a seeded
        offset in [0, needle_span), inside every block of the store."""
        rng = np.random.Generator(np.random.Philox(key=self.seed + 104729 * (b + 1)))
        return int(rng.integers(0, self.needle_span))

    def needle_at(self, unit: int, off_lo: int, n: int):
        """Offset (in the unit's tokens) of the needle inside [off_lo, off_lo + n) of stream
        unit `unit`, or None (not a store block, no needles, or outside the range)."""
        if self.needle_span <= 0 or unit < STORE_UNIT:
            return None
        t = self.needle_offset(unit - STORE_UNIT)
        return t if off_lo <= t < off_lo + n else None

    def seq_block(self, s: int, j: int) -> int:
        """Store block grafted into slot j of sequence s (window workloads).

        Slot j holds a block whose own position is j * block_tokens: the block id
        is drawn from {b : b mod blocks_per_seq == j} with a seeded choice.
        """
        n_choices = self.store_blocks // self.blocks_per_seq
        rng = np.random.Generator(np.random.Philox(key=self.seed + 7919 * (s + 1)))
        picks = rng.integers(0, n_choices, size=self.blocks_per_seq)
        return int(picks[j]) * self.blocks_per_seq + j

    def segments(self, s: int):
        """(logical t0, n_tokens, stream unit, token offset in that unit) covering
        sequence s's logical tokens [0, ctx_final)."""
        if self.fixed_unit >= 0:
            return [(0, self.ctx_final, self.fixed_unit, 0)]
        if self.explicit_segments:
            segs = [tuple(x) for x in self.explicit_segments]
            tail0 = segs[-1][0] + segs[-1][1]
            return segs + [(tail0, self.ctx_final - tail0, s, tail0)]
        if self.blocks_per_seq <= 1 or not self.block_tokens:
            return [(0, self.ctx_final, s, 0)]
        segs = []
        for j in range(self.blocks_per_seq):
            b = self.seq_block(s, j)
            segs.append((j * self.block_tokens, self.block_tokens, STORE_UNIT + b, 0))
        tail0 = self.blocks_per_seq * self.block_tokens
        segs.append((tail0, self.ctx_final - tail0, s, tail0))
        return segs


TINY = Workload(1, "tiny-f32", n_layers=1, n_q_heads=4, n_kv_heads=2, head_dim=64, dtype="f32",
                page_size=16, prefix=256, suffix=32, decode_steps=8, batch=1, sigma_log2=0)

BLOCK12B = Workload(2, "12b-block4096", n_layers=48, n_q_heads=16, n_kv_heads=8, head_dim=256,
                    dtype="bf16", page_size=16, prefix=4096, suffix=512, decode_steps=64, batch=1,
                    sigma_log2=-1)

WINDOW12B = Workload(3, "12b-window32k", n_layers=48, n_q_heads=16, n_kv_heads=8, head_dim=256,
                     dtype="bf16", page_size=16, prefix=32768, suffix=512, decode_steps=64, batch=16,
                     sigma_log2=-1, blocks_per_seq=8, block_tokens=4096, store_blocks=256,
                     store_tokens=256 * 4096)

RELOC31B = Workload(4, "31b-reloc16k", n_layers=60, n_q_heads=32, n_kv_heads=16, head_dim=128,
                    dtype="bf16", page_size=16, prefix=16384, suffix=1024, decode_steps=64, batch=8,
                    sigma_log2=-1, start_pos=8192, own_pos=0)

STORE12B = Workload(5, "12b-store2.85M", n_layers=48, n_q_heads=16, n_kv_heads=8, head_dim=256,
                    dtype="bf16", page_size=16, prefix=32768, suffix=35, decode_steps=8, batch=32,
                    sigma_log2=-1, blocks_per_seq=8, block_tokens=4096, store_blocks=697,
                    store_tokens=2_854_766, needle_span=2_854_766 - 696 * 4096)

NEEDLE_SIGMA_LOG2 = 0      # needle key and value rows: sigma 1

# the 12B-class block with Gemma-3-style attention: 1,024-key sliding windows on five of
# every six layers, the sixth global; the cache stays full-size for every layer (Sec. 4.3)
SWA12B = Workload(6, "12b-swa1024-block4096", n_layers=48, n_q_heads=16, n_kv_heads=8, head_dim=256,
                  dtype="bf16", page_size=16, prefix=4096, suffix=512, decode_steps=64, batch=1,
                  sigma_log2=-1, sliding_window=1024, global_every=6)

WORKLOADS = {w.wid: w for w in (TINY, BLOCK12B, WINDOW12B, RELOC31B, STORE12B, SWA12B)}


def scaled(w: Workload, **kw) -> Workload:
    """A smaller variant of a workload for parity tests (same dtype/head geometry)."""
    return dataclasses.replace(w, **kw)


def raw_rows(w: Workload, role: int, s: int, layers, t0: int, n: int):
    """Raw storage bits [len(layers)][n][H][D] for logical tokens [t0, t0+n) of sequence s."""
    from .philox import normal_tensor
    H = w.n_q_heads if role == ROLE_Q else w.n_kv_heads
    parts = []
    for (a, cnt, unit, off) in w.segments(s):
        lo, hi = max(a, t0), min(a + cnt, t0 + n)
        if lo >= hi:
            continue
        part = normal_tensor(w.seed, w.stream(role, unit), layers, off + (lo - a), hi - lo,
                             H, w.head_dim, w.sigma_log2, w.raw_dtype)
        tn = w.needle_at(unit, off + (lo - a), hi - lo) if role in (ROLE_K, ROLE_V) else None
        if tn is not None:
            part[:, tn - (off + (lo - a))] = needle_row(w, role, unit, layers)[:, 0]
        parts.append(part)
    return np.concatenate(parts, axis=1)


def needle_row(w: Workload, role: int, unit: int, layers):
    """The needle's raw key (role K) or value (role V) rows of store unit `unit`:
    bits [len(layers)][1][Hkv][D]."""
    from .philox import normal_tensor
    nrole = ROLE_NK if role == ROLE_K else ROLE_NV
    return normal_tensor(w.seed, w.stream(nrole, unit), layers, 0, 1, w.n_kv_heads, w.head_dim,
                         NEEDLE_SIGMA_LOG2, w.raw_dtype)


__all__ = ["Workload", "WORKLOADS", "TINY", "BLOCK12B", "WINDOW12B", "RELOC31B", "STORE12B",
           "scaled", "raw_rows", "needle_row", "ROLE_Q", "ROLE_K", "ROLE_V", "STORE_UNIT", "NEEDLE_SIGMA_LOG2"]
