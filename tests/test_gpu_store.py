"""Large-store paging on the GPU (Sec. 4.4): a 2,854,766-token store of 697 blocks (the last
one partial) streamed from host-pinned memory into a 32,768-token window of 8
direct-mapped slots shared by 32 decoding sequences.

Per access of block b at the paper's needle depths: graft from pinned host memory into
slot b mod 8 at the block's own position, a 35-token suffix prefill per sequence, 8 decode
steps.  Checked: the restored slot re-deposits to the artifact's exact bytes (the block
itself is the needle) while the other slots do not hold it (negative control: a window
parked elsewhere returns the wrong block); the access latency does not grow with depth;
the attention outputs after the last access match the oracle of the window's contents."""

import gc
import hashlib

import numpy as np
import pytest
import torch

from oracle.path import expected_rows
from synth.workloads import STORE12B

from gpu_helpers import attention_close

pytestmark = pytest.mark.gpu

DEPTH_BLOCKS = [0, 81, 169, 344, 520, 607, 688, 696]   # 0, 334k, 694k, 1.41M, 2.13M, 2.49M, 2.82M tokens + last


def _sha(t):
    return hashlib.sha256(t.contiguous().view(torch.uint8).cpu().numpy().tobytes()).hexdigest()


def test_store_depth_sweep():
    from paper_2607_14431_amd import harness as h
    w = STORE12B
    assert (w.store_blocks - 1) * w.block_tokens + w.store_block_tokens(w.store_blocks - 1) == w.store_tokens
    win = h.StoreWindow(w)
    full_bytes = h.kvg.kvg_payload_bytes(win.cache, w.block_tokens)
    pinned = h.PinnedPayload(full_bytes)
    print("store: initial window fill, blocks 0..7", flush=True)
    for b in range(win.slots):
        hdr = win.materialize(b, pinned)
        win.graft(b, hdr, pinned)
        torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    rows = []
    res = None
    for b in DEPTH_BLOCKS:
        hdr = win.materialize(b, pinned)              # the store's deposit of block b (untimed)
        art_sha = hashlib.sha256(pinned.host[: hdr.payload_bytes].numpy().tobytes()).hexdigest()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        win.graft(b, hdr, pinned)
        ev[1].record(stream)
        win.arm.w = win.view()
        suf = h.prefill(win.arm, win.win_tokens, w.suffix)
        ev[2].record(stream)
        dec = h.decode(win.arm, win.win_tokens + w.suffix, w.decode_steps)
        ev[3].record(stream)
        torch.cuda.synchronize()
        t = [ev[i].elapsed_time(ev[i + 1]) for i in range(3)]
        j = b % win.slots
        _, slot_bytes = h.deposit(win.arm, 0, j * w.block_tokens, hdr.n_tokens, j * w.block_tokens)
        _, other = h.deposit(win.arm, 0, ((j + 1) % win.slots) * w.block_tokens, hdr.n_tokens,
                             ((j + 1) % win.slots) * w.block_tokens)
        assert _sha(slot_bytes) == art_sha, f"block {b}: restored slot differs from the artifact"
        assert _sha(other) != art_sha, f"block {b}: negative control found the block in another slot"
        gbps = hdr.payload_bytes / (t[0] * 1e-3) / 1e9
        rows.append((b, b * w.block_tokens, t[0], t[1], t[2], gbps))
        print(f"store access block {b:3d} (depth {b * w.block_tokens:>9,d} tokens): graft from host {t[0]:7.2f} ms "
              f"({gbps:5.1f} GB/s), suffix prefill x{win.batch} {t[1]:7.2f} ms, {w.decode_steps} decode steps "
              f"x{win.batch} {t[2]:7.2f} ms", flush=True)
        res = (suf, dec)
        del slot_bytes, other

    full = [r for r in rows if r[0] != w.store_blocks - 1]
    g = [r[2] for r in full]
    assert max(g) < 2.0 * min(g), f"graft latency grows with depth: {g}"

    print("store: oracle on the window after the last access", flush=True)
    vw = win.view()
    suf, dec = res
    for s in (0, win.batch - 1):
        r_idx = [0, 17, w.suffix - 1]
        st_idx = [0, w.decode_steps - 1]
        want = expected_rows(vw, s, [0], [vw.prefix + r for r in r_idx] + [vw.prefix + w.suffix + t for t in st_idx])[0]
        got = np.concatenate([suf[0, s, r_idx].cpu().numpy(), dec[st_idx, 0, s].cpu().numpy()], axis=0)
        print("store oracle seq", s, attention_close(got.astype(np.float64), want, w.dtype))
    del win, pinned
    gc.collect()
    torch.cuda.empty_cache()
