"""Logit head and logit comparison on the GPU against the oracle, and the paper's logit-level
verdict on a graft (Eq. 1-2, Sec. 4.1's table): 50 samples of graft against fresh with SHA-256
equality of every logit row, zero KL, equal argmax, and the Mann-Whitney test against the
noise floor (p = 1, Cliff's delta 0); a relocated graft (Sec. 4.2) as the contrast, whose KLs
are small but nonzero and stand apart from the floor."""

import numpy as np
import pytest
import torch

from oracle.logits import argmax as o_argmax
from oracle.logits import kl_divergence, log_softmax, logit_head
from oracle.numerics import bits_to_values
from synth import ROLE_H, ROLE_W, Stream, normal_tensor
from synth.workloads import BLOCK12B, RELOC31B, scaled

pytestmark = pytest.mark.gpu

WID = 40            # generator stream family of these standalone cases


def _hidden(rows, H, sig=-1):
    bits = normal_tensor(5, Stream(WID, ROLE_H, 0), [0], 0, rows, 1, H, sig, "f32")[0, :, 0]
    return bits.view(np.float32)


def _weights(V, H, sig=-2, v0=0):
    return normal_tensor(5, Stream(WID, ROLE_W, 0), [0], v0, V, 1, H, sig, "bf16")[0, :, 0]


def _tolerance(hidden, w_vals, want, H):
    """fp32 accumulation of H products in any order: |error| <= gamma_H sum_k |h_k w_k|
    (gamma_n = n u / (1 - n u), u = 2^-24); the soft cap has slope <= 1 and tanhf, the
    division and the multiply add a few units in the last place of the result."""
    from oracle.numerics import round_bf16
    h = np.abs(round_bf16(hidden.astype(np.float64)))
    s = h @ np.abs(w_vals).T
    u = 2.0 ** -24
    return H * u / (1 - H * u) * s + 2.0 ** -20 * np.abs(want) + 1e-30


CASES = [
    # rows, H, V, cap
    (5, 256, 1003, 30.0),      # V not a multiple of 4 or of a workgroup's 512 rows
    (40, 4096, 8292, 30.0),    # two row tiles, the second ragged
    (1, 128, 600, 0.0),        # no soft cap, smallest hidden size
    (33, 512, 512, 50.0),      # 33..64 rows: two row tiles per wave
    (100, 256, 700, 30.0),     # 65..128 rows: four row tiles per wave
    (130, 128, 300, 30.0),     # past 128 rows: a second read of W
]


@pytest.mark.parametrize("rows,H,V,cap", CASES)
def test_logits_match_oracle(rows, H, V, cap):
    from paper_2607_14431_amd import kvg
    hid = _hidden(rows, H)
    wb = _weights(V, H)
    w_vals = bits_to_values(wb, "bf16")
    from paper_2607_14431_amd import harness as h
    head = h.pack_head(torch.from_numpy(wb.view(np.int16)).cuda().view(torch.bfloat16))
    out = torch.full((rows, V), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(kvg.kvg_logits_workspace_bytes(rows, H), dtype=torch.uint8, device="cuda")
    kvg.kvg_logits(torch.from_numpy(hid).cuda(), head.packed, V, cap, out, ws)
    got = out.cpu().numpy().astype(np.float64)
    want = logit_head(hid, w_vals, cap)
    tol = _tolerance(hid, w_vals, want, H)
    err = np.abs(got - want)
    print(f"rows {rows} H {H} V {V}: max err {err.max():.3e}, max tol {tol.max():.3e}, max |logit| {np.abs(want).max():.2f}")
    assert np.all(np.isfinite(got))
    assert np.all(err <= tol)
    if cap:
        assert np.abs(want).max() > 0.2 * cap     # the cap is exercised


def test_logits_full_vocabulary_sampled():
    """50 rows x 262,144 vocabulary rows x 4,096 (two row tiles), oracle on sampled rows."""
    from paper_2607_14431_amd import harness as h
    rows, H, V = 50, 4096, 262_144
    w = scaled(BLOCK12B)
    sig = -2                                      # with unit-scale hidden values: logits up to ~25
    wt = h.head_weights(w, sigma_log2=sig)
    hid = _hidden(rows, H)
    out = h.logits(torch.from_numpy(hid).cuda(), wt)
    again = h.logits(torch.from_numpy(hid).cuda(), wt)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int32), again.view(torch.int32)), "not deterministic"
    rng = np.random.default_rng(11)
    vs = np.unique(np.concatenate([np.arange(64), np.arange(V - 64, V), rng.integers(0, V, 512)]))
    w_vals = np.stack([bits_to_values(normal_tensor(w.seed, w.stream(ROLE_W, 0), [0], int(v), 1, 1, H,
                                                    sig, "bf16")[0, 0, 0], "bf16") for v in vs])
    want = logit_head(hid, w_vals, h.HEAD_CAP)
    got = out[:, torch.from_numpy(vs).cuda()].cpu().numpy().astype(np.float64)
    tol = _tolerance(hid, w_vals, want, H)
    print(f"full vocabulary: max err {np.abs(got - want).max():.3e}, max |logit| {np.abs(want).max():.2f}")
    assert np.all(np.abs(got - want) <= tol)


def test_logit_compare_matches_oracle():
    from paper_2607_14431_amd import harness as h
    rows, V = 6, 100_003
    rng = np.random.default_rng(2)
    a = (rng.normal(size=(rows, V)) * 6).astype(np.float32)
    b = (a + rng.normal(size=(rows, V)) * np.array([0, 1e-3, 1e-2, 0.1, 1.0, 3.0])[:, None]).astype(np.float32)
    a[0, [7, 99_000]] = a[0].max() + 1.0          # tied maximum: the first index wins
    b[0] = a[0]                                    # byte-equal row: KL exactly 0
    kl, ia, ib = h.compare_logits(torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda())
    want = kl_divergence(a.astype(np.float64), b.astype(np.float64))
    # fp64 sums of V terms p_i (la_i - lb_i) in another order: |error| <= gamma_V sum |terms|
    # (with a margin of 4 for the log-sum-exp's own rounding), u = 2^-53
    la, lb = log_softmax(a), log_softmax(b)
    tol = 4 * V * 2.0 ** -53 * (np.exp(la) * np.abs(la - lb)).sum(axis=1)
    print("kl", kl, "oracle", want, "diff", np.abs(kl - want), "tol", tol)
    assert kl[0] == 0.0 and ia[0] == 7
    assert np.all(np.abs(kl - want) <= tol)
    assert np.array_equal(ia, o_argmax(a)) and np.array_equal(ib, o_argmax(b))


def _arms(h, w, trial, relocate_to=None):
    """(fresh, graft) results of one trial; the graft is relocated to `relocate_to` if given."""
    fresh = h.new_arm(w, [0], w.ctx_final, seed=300 + trial, poison_id=0, spare_pages=3)
    h.fresh_prefix(fresh)
    hdr, payload = h.deposit(fresh, 0, 0, w.prefix, fresh.start_pos)
    rf = h.continue_arm(fresh)
    target = fresh.start_pos if relocate_to is None else relocate_to
    gw = w if relocate_to is None else scaled(w, start_pos=relocate_to)
    g = h.new_arm(gw, [0], w.ctx_final, seed=400 + trial, poison_id=1, start_pos=target, spare_pages=5)
    h.graft(g, 0, hdr, payload, 0, target, relocate=relocate_to is not None)
    rg = h.continue_arm(g)
    return rf, rg


def test_graft_logit_verdict_fifty_samples():
    """Sec. 4.1's table on the 12B-class geometry: 50 samples (40 suffix rows and 10 decode
    steps of the last layer), graft vs fresh, noise floor fresh vs a second fresh run."""
    from paper_2607_14431_amd import harness as h
    w = scaled(BLOCK12B, n_layers=4, prefix=1100, suffix=40, decode_steps=10)
    rf, rg = _arms(h, w, 0)
    rf2 = h.continue_arm(_fresh_again(h, w))
    wt = h.head_weights(w)
    lf, lg, ln = (h.logits(h.hidden_rows(r, 0), wt) for r in (rf, rg, rf2))
    st = h.exactness_stats(lg, lf, ln)
    print(st)
    assert st["samples"] == 50 and st["sha256_equal"] == 50
    assert st["kl_median"] == 0.0 and st["kl_p99"] == 0.0 and st["argmax_disagree"] == 0
    assert st["noise_kl_median"] == 0.0 and st["mann_whitney_p"] == 1.0 and st["cliffs_delta"] == 0.0
    # the logits are spread over the soft cap's range, not collapsed near 0
    assert lf.abs().max().item() > 10.0


def _fresh_again(h, w):
    arm = h.new_arm(w, [0], w.ctx_final, seed=999, poison_id=1, spare_pages=9)
    h.fresh_prefix(arm, chunk=256)               # a different chunking of the same prefix
    return arm


def test_relocated_graft_logits_differ_from_floor():
    """Relocation by +8192 (Sec. 4.2): every sample's logits differ from the fresh computation
    at the new offset, their KLs are small and all above the zero floor (Cliff's delta 1)."""
    from paper_2607_14431_amd import harness as h
    d = 8192
    w0 = scaled(RELOC31B, n_layers=2, prefix=600, suffix=40, decode_steps=10, batch=1, start_pos=0)
    _, rg = _arms(h, w0, 1, relocate_to=d)
    wd = scaled(w0, start_pos=d)
    fresh_d = h.new_arm(wd, [0], wd.ctx_final, seed=501, poison_id=0)
    h.fresh_prefix(fresh_d)
    rfd = h.continue_arm(fresh_d)
    fresh_d2 = h.new_arm(wd, [0], wd.ctx_final, seed=502, poison_id=1)
    h.fresh_prefix(fresh_d2)
    rfd2 = h.continue_arm(fresh_d2)
    wt = h.head_weights(w0)
    lg, lf, ln = (h.logits(h.hidden_rows(r, 0), wt) for r in (rg, rfd, rfd2))
    st = h.exactness_stats(lg, lf, ln)
    print(st)
    assert st["sha256_equal"] < st["samples"]
    assert 0.0 < st["kl_median"] < 0.1
    assert st["noise_kl_median"] == 0.0 and st["mann_whitney_p"] < 1e-6 and st["cliffs_delta"] > 0.9
