"""Decode steps captured in a HIP graph and replayed.

The library launches on the caller's stream and allocates nothing, so a caller can capture its
calls (here with torch.cuda.CUDAGraph, which captures the launches the library makes on the
capture stream) and replay them; the allocation-free decode entry point exists for such
callers.  A graph of several consecutive decode steps (each step's raw rows in buffers of its
own, each step appending its token) is replayed several times with eager work and
synchronisations between the replays, and every replay must give the bytes of the eager calls:
outputs and cache pages.  The workspace entry point is captured the same way."""

import numpy as np
import pytest
import torch

from synth import ROLE_K, ROLE_Q, ROLE_V
from synth.gpu import raw_chunk
from synth.workloads import BLOCK12B, scaled

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("noalloc", [True, False], ids=["noalloc", "workspace"])
def test_decode_graph_replays_match_eager(noalloc):
    from paper_2607_14431_amd import harness as h
    from paper_2607_14431_amd import kvg

    w = scaled(BLOCK12B, n_layers=3, prefix=1100, suffix=1, decode_steps=4, sliding_window=700, global_every=3)
    N, T, B = w.prefix, w.decode_steps, 2
    arm = h.new_arm(w, [0, 1], N + T, seed=21, poison_id=0)
    h.prefill(arm, 0, N, append_only=True)
    rp = h.rope_of(w)
    metas = [arm.meta(N + i) for i in range(T)]
    rows = [tuple(raw_chunk(w, r, arm.seqs, N + i, 1)[:, :, 0].contiguous() for r in (ROLE_Q, ROLE_K, ROLE_V))
            for i in range(T)]
    ws = kvg.decode_workspace(arm.cache, metas[-1], w.n_layers)

    def steps(out):
        for i in range(T):
            q, k, v = rows[i]
            if noalloc:
                kvg.kvg_decode_attn_noalloc(arm.cache, metas[i], rp, 0, w.n_layers, q, k, v, w.scale, out[i])
            else:
                kvg.kvg_decode_attn(arm.cache, metas[i], rp, 0, w.n_layers, q, k, v, w.scale, out[i], ws)

    shape = (T, w.n_layers, B, w.n_q_heads, w.head_dim)
    eager = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
    steps(eager)                          # also takes the fixed workspace's address, outside capture
    torch.cuda.synchronize()
    pages = arm.cache.k_pool.clone(), arm.cache.v_pool.clone()
    assert torch.isfinite(eager).all()

    out = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        steps(out)
    torch.cuda.synchronize()
    for rep in range(4):
        out.fill_(float("nan"))                                # eager work between the replays
        scratch = torch.randn(1 << 20, device="cuda").sum()    # noqa: F841
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int32), eager.view(torch.int32)), f"replay {rep} differs from eager"
        assert torch.equal(arm.cache.k_pool.view(torch.int16), pages[0].view(torch.int16))
        assert torch.equal(arm.cache.v_pool.view(torch.int16), pages[1].view(torch.int16))
    del graph
    assert np.isfinite(out.cpu().numpy()).all()
