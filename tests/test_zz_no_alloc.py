"""kvg_decode_attn_noalloc (the decode call on the library's own fixed workspace, for callers
that cannot allocate) gives the same bytes as kvg_decode_attn on a caller's workspace: two
calls in a row through the C ABI, the second with a smaller batch and shorter contexts, and
a call whose workspace would exceed the fixed array is refused before anything runs."""

import numpy as np
import pytest
import torch

from synth import ROLE_K, ROLE_Q, ROLE_V, normal_tensor
from synth.philox import Stream

from gpu_helpers import bits_to_device

pytestmark = pytest.mark.gpu


def _gen(role, s, t0, n, L, H, D):
    return normal_tensor(91, Stream(60, role, s), range(L), t0, n, H, D, -1, "bf16")


def _case(kvg, L, Hq, Hkv, D, ctxs, windows=None):
    """A bf16 cache holding each sequence's context, and one decode step's raw rows."""
    B = len(ctxs)
    per_seq = (max(ctxs) + 1 + 15) // 16
    n_pages = B * per_seq + 2
    tables = np.random.default_rng(sum(ctxs)).permutation(n_pages)[: B * per_seq].reshape(B, per_seq).astype(np.int32)
    cache = kvg.Cache.allocate(L, n_pages, Hq, Hkv, D, torch.bfloat16, windows=windows)
    cache.k_pool.view(torch.int16).fill_(0x7FC1)
    cache.v_pool.view(torch.int16).fill_(0x7FC1)
    tb = torch.from_numpy(tables).cuda()
    st = torch.tensor([5 * b for b in range(B)], dtype=torch.int64, device="cuda")
    rp = kvg.rope(10000.0)
    for b, c in enumerate(ctxs):
        one = kvg.Seqs(tb[b:b + 1], torch.zeros(1, dtype=torch.int32, device="cuda"), st[b:b + 1], 0)
        kvg.kvg_append(cache, one, rp, 0, L, c, bits_to_device(_gen(ROLE_K, b, 0, c, L, Hkv, D)[:, None], "bf16"),
                       bits_to_device(_gen(ROLE_V, b, 0, c, L, Hkv, D)[:, None], "bf16"))
    raw = [bits_to_device(np.ascontiguousarray(np.stack([_gen(r, b, c, 1, L, H, D)[:, 0] for b, c in enumerate(ctxs)],
                                                        axis=1)), "bf16")
           for r, H in ((ROLE_Q, Hq), (ROLE_K, Hkv), (ROLE_V, Hkv))]
    seqs = kvg.Seqs(tb, torch.tensor(ctxs, dtype=torch.int32, device="cuda"), st, max(ctxs))
    return cache, seqs, rp, raw


def _both(kvg, cache, seqs, rp, raw, L, Hq, D):
    """The decode step through both entry points, each on its own copy of the cache (the step
    appends the new token, so the two calls must not share it)."""
    B = seqs.block_tables.shape[0]
    outs = []
    for noalloc in (False, True):
        c = kvg.Cache(cache.k_pool.clone(), cache.v_pool.clone(), cache.n_q_heads, cache.windows)
        out = torch.full((L, B, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
        if noalloc:
            kvg.kvg_decode_attn_noalloc(c, seqs, rp, 0, L, *raw, 1.0 / np.sqrt(D), out)
        else:
            kvg.kvg_decode_attn(c, seqs, rp, 0, L, *raw, 1.0 / np.sqrt(D), out, kvg.decode_workspace(c, seqs, L))
        torch.cuda.synchronize()
        outs.append((out, c))
    return outs


def test_noalloc_decode_matches_workspace_decode():
    from paper_2607_14431_amd import kvg
    L, Hq, Hkv, D = 3, 8, 4, 256
    # first call: 5 sequences, contexts across several 512-key splits and a windowed layer
    cache, seqs, rp, raw = _case(kvg, L, Hq, Hkv, D, [3000, 17, 1024, 2600, 511], windows=(0, 700, 0))
    (o_ws, c_ws), (o_na, c_na) = _both(kvg, cache, seqs, rp, raw, L, Hq, D)
    assert torch.isfinite(o_na).all()
    assert torch.equal(o_ws.view(torch.int32), o_na.view(torch.int32))
    assert torch.equal(c_ws.k_pool.view(torch.int16), c_na.k_pool.view(torch.int16))   # the same token appended
    # second call: smaller batch and contexts (the array keeps the first call's partials)
    cache2, seqs2, rp2, raw2 = _case(kvg, L, Hq, Hkv, D, [700, 40])
    (o_ws2, _), (o_na2, _) = _both(kvg, cache2, seqs2, rp2, raw2, L, Hq, D)
    assert torch.isfinite(o_na2).all()
    assert torch.equal(o_ws2.view(torch.int32), o_na2.view(torch.int32))
    # a call needing more workspace than the array holds is refused before anything runs
    # (a 1.2M-token bound over 5 sequences: 2,344 splits of partials per row-head; the table only
    # has to be long enough for the bound, the call never reads it)
    wide = torch.zeros((5, 75_008), dtype=torch.int32, device="cuda")
    big = kvg.Seqs(wide, seqs.ctx_lens, seqs.start_pos, 1_200_000)
    assert kvg.kvg_decode_workspace_bytes(cache, big, L) > kvg.KVG_NOALLOC_SCRATCH_BYTES
    with pytest.raises(kvg.KvgError) as e:
        kvg.kvg_decode_attn_noalloc(cache, big, rp, 0, L, *raw, 1.0 / np.sqrt(D), o_na)
    assert e.value.name == "KVG_E_WORKSPACE"
