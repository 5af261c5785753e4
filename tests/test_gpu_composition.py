"""Sequential composition and chunk invariance on the GPU.

The paper finds that a chunked prefill and a monolithic prefill of the same tokens give
different bytes in its engine, so its sequential composition (graft A, prefill B on top) is
byte-exact only against a chunked reference (Sec. 4.2, 4.8).  Here every reduction is
ordered by logical key index alone (prefill key tiles at absolute multiples of 64, decode splits at
absolute multiples of 512), so:

  * a prefill in ragged chunks produces the same bytes as one monolithic prefill: the
    attention outputs of every row, the cache contents (deposited and hashed) and the decode
    steps that follow;
  * sequential composition holds: graft A at [0, |A|), prefill B on top in chunks, deposit
    A || B, and the result equals the fresh monolithic computation of A || B byte for byte.

Covered paths: bf16 MFMA prefill (group 2, D 256 and 128), bf16 VALU prefill (group 8),
fp32 VALU prefill and fp8 caches, each also with sliding-window layers beside global ones (a windowed row
skips the key tiles and decode splits below its window, which depend on where its chunk
starts; the bytes must not).  Chunk sizes cross page (16) and key-tile (64) boundaries."""

import hashlib

import pytest
import torch

from synth.workloads import BLOCK12B, TINY, scaled

pytestmark = pytest.mark.gpu

A, B = 1000, 300                       # |A| = 15 tiles of 64 + 40; |A| + |B| = 1300
CHUNKS = [1, 63, 65, 300, 571, 300]    # ragged split of [0, 1300)
STEPS = 4

GEOMS = {
    "bf16-mfma-d256-g2": scaled(BLOCK12B, n_layers=3, prefix=A, suffix=B, decode_steps=STEPS),
    "bf16-mfma-d128-g2": scaled(BLOCK12B, n_layers=2, n_q_heads=8, n_kv_heads=4, head_dim=128,
                                prefix=A, suffix=B, decode_steps=STEPS),
    "bf16-valu-d128-g8": scaled(BLOCK12B, n_layers=2, n_q_heads=16, n_kv_heads=2, head_dim=128,
                                prefix=A, suffix=B, decode_steps=STEPS),
    "f32-valu-d64-g2": scaled(TINY, n_layers=2, prefix=A, suffix=B, decode_steps=STEPS),
    # two windowed layers and a global one; windows end inside a key tile and a page
    "swa-bf16-mfma-d256-g2": scaled(BLOCK12B, n_layers=3, prefix=A, suffix=B, decode_steps=STEPS,
                                    sliding_window=200, global_every=3),
    "swa-bf16-valu-d128-g8": scaled(BLOCK12B, n_layers=3, n_q_heads=16, n_kv_heads=2, head_dim=128,
                                    prefix=A, suffix=B, decode_steps=STEPS, sliding_window=555, global_every=2),
    "swa-f32-valu-d64-g2": scaled(TINY, n_layers=2, prefix=A, suffix=B, decode_steps=STEPS,
                                  sliding_window=77, global_every=2),
    # fp8 E4M3 cache (bf16 inputs rounded once when stored)
    "fp8-valu-d256-g2": scaled(BLOCK12B, n_layers=2, prefix=A, suffix=B, decode_steps=STEPS, dtype="fp8"),
}


@pytest.fixture(scope="module")
def h():
    from paper_2607_14431_amd import harness
    return harness


def _sha(t):
    return hashlib.sha256(t.contiguous().view(torch.uint8).cpu().numpy().tobytes()).hexdigest()


def _chunked(h, arm, t0, sizes):
    outs, t = [], t0
    for n in sizes:
        outs.append(h.prefill(arm, t, n))
        t += n
    return torch.cat(outs, dim=2), t


@pytest.mark.parametrize("name", list(GEOMS))
def test_chunked_prefill_equals_monolithic(h, name):
    w = GEOMS[name]
    n = A + B
    assert sum(CHUNKS) == n
    print(f"composition {name}: monolithic arm", flush=True)
    mono = h.new_arm(w, [0], w.ctx_final, seed=700, poison_id=0)
    out_m = h.prefill(mono, 0, n)
    dec_m = h.decode(mono, n, STEPS)
    print(f"composition {name}: chunked arm {CHUNKS}", flush=True)
    chk = h.new_arm(w, [0], w.ctx_final, seed=701, poison_id=1)
    out_c, t = _chunked(h, chk, 0, CHUNKS)
    assert t == n
    dec_c = h.decode(chk, n, STEPS)
    torch.cuda.synchronize()
    assert h.bytes_equal(out_c, out_m), "chunked prefill outputs differ from the monolithic prefill"
    assert h.bytes_equal(dec_c, dec_m), "decode after chunked prefill differs"
    _, dep_m = h.deposit(mono, 0, 0, n + STEPS, 0)
    _, dep_c = h.deposit(chk, 0, 0, n + STEPS, 0)
    assert _sha(dep_m) == _sha(dep_c), "cache contents differ"


@pytest.mark.parametrize("name", ["bf16-mfma-d256-g2", "f32-valu-d64-g2", "swa-bf16-mfma-d256-g2", "fp8-valu-d256-g2"])
def test_sequential_composition(h, name):
    """graft A, prefill B on top (chunked), deposit A || B == fresh monolithic A || B."""
    w = GEOMS[name]
    n = A + B
    print(f"composition {name}: fresh monolithic A || B", flush=True)
    mono = h.new_arm(w, [0], w.ctx_final, seed=710, poison_id=0)
    out_m = h.prefill(mono, 0, n)
    dec_m = h.decode(mono, n, STEPS)
    _, dep_m = h.deposit(mono, 0, 0, n, 0)

    print(f"composition {name}: capture A", flush=True)
    src = h.new_arm(w, [0], w.ctx_final, seed=711, poison_id=1)
    _chunked(h, src, 0, [A])
    hdr, art = h.deposit(src, 0, 0, A, 0)

    print(f"composition {name}: graft A, prefill B in chunks", flush=True)
    g = h.new_arm(w, [0], w.ctx_final, seed=712, poison_id=1)
    h.graft(g, 0, hdr, art, 0, 0)
    out_b, t = _chunked(h, g, A, [7, 57, 236])
    assert t == n
    dec_g = h.decode(g, n, STEPS)
    _, dep_g = h.deposit(g, 0, 0, n, 0)
    torch.cuda.synchronize()
    assert _sha(dep_g) == _sha(dep_m), "deposit of A || B differs from the fresh computation"
    assert h.bytes_equal(out_b, out_m[:, :, A:]), "B's rows differ from the fresh computation"
    assert h.bytes_equal(dec_g, dec_m), "decode after composition differs"


def test_window_past_context_is_full_attention(h):
    """A window at least as long as every row's causal prefix selects every key: the bytes
    equal those of the same layers without a window (one code path, same reduction order)."""
    base = GEOMS["bf16-mfma-d256-g2"]
    wide = scaled(base, sliding_window=A + B + STEPS, global_every=0)
    outs = []
    for w in (base, wide):
        arm = h.new_arm(w, [0], w.ctx_final, seed=720, poison_id=0)
        out = h.prefill(arm, 0, A + B)
        outs.append((out, h.decode(arm, A + B, STEPS)))
    torch.cuda.synchronize()
    assert h.bytes_equal(outs[0][0], outs[1][0])
    assert h.bytes_equal(outs[0][1], outs[1][1])
