"""Byte-exact graft (Sec. 3.2, Eq. 1) on the GPU through the C ABI.

graft == fresh: the suffix-prefill and decode outputs computed on a grafted cache are
byte-identical to those computed on the freshly prefilled cache (different physical page
permutation and poison in the two caches).  fresh == fresh across trials is the
self-comparison floor.  The restored pages re-deposit to the artifact's exact bytes.
Relocation (Sec. 4.2) is not byte-exact: its residual against a fresh computation at the
new offset is reported and the relocated outputs still match the oracle.
"""

import hashlib

import numpy as np
import pytest
import torch

from oracle.path import expected_rows, relocated_kv
from synth.workloads import BLOCK12B, RELOC31B, TINY, scaled

from gpu_helpers import attention_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def h():
    from paper_2607_14431_amd import harness
    return harness


def _sha(t):
    return hashlib.sha256(t.contiguous().view(torch.uint8).cpu().numpy().tobytes()).hexdigest()


def run_pair(h, w, trial, seqs=None, graft_start=None, relocate=False, prefix_mode="prefill"):
    """Fresh arm and graft arm of one trial; returns (fresh result, graft result, payload shas)."""
    seqs = list(range(w.batch)) if seqs is None else seqs
    fresh = h.new_arm(w, seqs, w.ctx_final, seed=100 + trial, poison_id=0, spare_pages=7)
    h.fresh_prefix(fresh, append_only=(prefix_mode == "append"))
    arts = [h.deposit(fresh, bi, 0, w.prefix, fresh.start_pos) for bi in range(len(seqs))]
    res_fresh = h.continue_arm(fresh)
    target = fresh.start_pos if graft_start is None else graft_start
    gw = w if graft_start is None else scaled(w, start_pos=graft_start)
    g = h.new_arm(gw, seqs, w.ctx_final, seed=200 + trial, poison_id=1, start_pos=target, spare_pages=3)
    for bi, (hdr, payload) in enumerate(arts):
        h.graft(g, bi, hdr, payload, 0, target, relocate=relocate)
    restored = [h.deposit(g, bi, 0, w.prefix, target)[1] for bi in range(len(seqs))]
    res_graft = h.continue_arm(g)
    torch.cuda.synchronize()
    shas = [(_sha(p), _sha(r)) for (_, p), r in zip(arts, restored)]
    return res_fresh, res_graft, shas


def _oracle_check(w, res, seqs, kv=None):
    rows = list(range(w.prefix, w.ctx_final))
    worst = (0.0, 0.0)
    for bi, s in enumerate(seqs):
        want = expected_rows(w, s, range(w.n_layers), rows, kv=None if kv is None else kv[bi])
        got = np.concatenate([res.suffix[:, bi].cpu().numpy(),
                              np.moveaxis(res.decode[:, :, bi].cpu().numpy(), 0, 1)], axis=1).astype(np.float64)
        worst = max(worst, attention_close(got, want, w.dtype))
    return worst


def test_tiny_graft_equals_fresh_five_trials(h):
    w = TINY
    digests = set()
    for trial in range(5):
        rf, rg, shas = run_pair(h, w, trial)
        for art, restored in shas:
            assert art == restored, "restored pages differ from the artifact"
        df, dg = rf.digest(), rg.digest()
        assert df == dg, f"trial {trial}: graft != fresh"
        digests.add(df)
    assert len(digests) == 1, "fresh runs are not bit-identical across trials"
    _oracle_check(w, rf, [0])


@pytest.mark.parametrize("w", [scaled(BLOCK12B, n_layers=3, prefix=1024, suffix=96, decode_steps=3),
                               scaled(RELOC31B, n_layers=2, prefix=1040, suffix=64, decode_steps=2, batch=2,
                                      start_pos=0),
                               scaled(BLOCK12B, n_layers=3, prefix=1024, suffix=96, decode_steps=3, dtype="fp8")],
                         ids=["12b-geom", "31b-geom", "12b-geom-fp8"])
def test_bf16_graft_equals_fresh(h, w):
    rf, rg, shas = run_pair(h, w, 0)
    assert all(a == r for a, r in shas)
    assert h.bytes_equal(rf.suffix, rg.suffix) and h.bytes_equal(rf.decode, rg.decode)
    _oracle_check(w, rg, list(range(w.batch)))


def test_batch_invariance(h):
    """Sequence 1 computed alone equals sequence 1 computed in a batch of 3 (byte for byte)."""
    w = scaled(BLOCK12B, n_layers=2, prefix=700, suffix=40, decode_steps=2, batch=3)
    rf, rg, _ = run_pair(h, w, 1)
    w1 = scaled(w, batch=1)
    rf1, rg1, _ = run_pair(h, w1, 2, seqs=[1])
    assert h.bytes_equal(rg.suffix[:, 1], rg1.suffix[:, 0])
    assert h.bytes_equal(rg.decode[:, :, 1], rg1.decode[:, :, 0])


def test_relocation_residual_reported(h):
    """Own position is byte-exact; relocation by +d is not (Sec. 4.2) but stays within the
    oracle tolerance; the graft-free control (fresh at 0 vs fresh at d) differs likewise."""
    d = 8192
    w0 = scaled(RELOC31B, n_layers=2, prefix=512, suffix=48, decode_steps=2, batch=1, start_pos=0)
    rf0, rg0, _ = run_pair(h, w0, 3)
    assert h.bytes_equal(rf0.suffix, rg0.suffix) and h.bytes_equal(rf0.decode, rg0.decode)
    # relocated: block captured at 0, grafted at d; reference: fresh at d
    _, rg_d, _ = run_pair(h, w0, 3, graft_start=d, relocate=True)
    wd = scaled(w0, start_pos=d)
    fresh_d, _, _ = run_pair(h, wd, 4)
    assert not h.bytes_equal(rg_d.suffix, fresh_d.suffix)
    res = (rg_d.suffix - fresh_d.suffix).abs().max().item()
    ctrl = (rf0.suffix - fresh_d.suffix).abs().max().item()
    print(f"relocation residual max-abs {res:.3e}; graft-free control {ctrl:.3e}")
    # the relocated outputs match the oracle of the relocated cache contents
    kv = [relocated_kv(scaled(w0, start_pos=d, own_pos=0), 0, range(w0.n_layers), w0.prefix, w0.ctx_final)]
    _oracle_check(scaled(w0, start_pos=d), rg_d, [0], kv=kv)
