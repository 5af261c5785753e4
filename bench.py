"""Benchmark of the byte-exact KV grafting hot path on one MI355X.

One step = the whole hot path over one batch of synthetic input, all inputs already
resident in HBM: deposit of the prefix block (gather), graft of the artifact into a
second cache at its own position (scatter), suffix chunked-prefill attention on the
grafted cache, then every decode step.  Workload: the 12B-class single-block case (48
layers, 16 query / 8 KV heads, head_dim 256, bf16, one 4,096-token block, 512-token
suffix, 64 decode steps, batch 1).

Prints one JSON line.  `value` is the graft restore rate (payload bytes read + pool bytes
written, per graft launch time); decode tokens/s and its HBM fraction, the graft==fresh
verdict (outside the timed region), per-phase times, the roofline of the dominant kernel
and the oracle's CPU baseline are reported beside it.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, vendor figure
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA, vendor figure
# 32-bit VALU lane operations per second: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
VALU_PEAK_GOPS = 256 * 4 * 16 * 2.4
SHA256_OPS_PER_BLOCK = 1401     # VALU lane operations per 64-byte block of the leaf-digest kernel


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-verify", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the figures taken after the timed steps (content digests, sliding-window "
                        "launches), so that a counter pass sees only the step's kernels")
    p.add_argument("--workload", default="12b-block4096",
                   choices=["12b-block4096", "12b-window32k", "31b-reloc16k", "12b-store2.85M"],
                   help="12b-block4096 (default) times the step; the other two time the full-size 32k-window "
                        "(batch 16) and 31B relocated (batch 8) configurations phase by phase")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 1 GiB device-to-device copy three times (the reference dispatch "
                        "that scales the FETCH_SIZE / WRITE_SIZE counters to bytes) and exit")
    return p.parse_args()


def copy_calibration():
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "dispatches": 3}), flush=True)


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "traffic_12b_block4096.md")


def measured_traffic(key: str):
    """HBM bytes per launch of a kernel as counted by rocprofv3 (FETCH_SIZE + WRITE_SIZE,
    scaled by a plain copy's counts) in the committed traffic summary, or None when the
    summary is absent or the kernel's sources have changed since the counters were taken."""
    try:
        text = open(TRAFFIC_PROFILE).read()
    except OSError:
        return None
    kv = {}
    for ln in text.splitlines():
        if " = " in ln:
            k, v = ln.strip().split(" = ", 1)
            kv[k] = v
    if key not in kv or "sources" not in kv:
        return None
    h = hashlib.sha256()
    for rel in kv["sources"].split():
        try:
            h.update(open(os.path.join(ROOT, rel), "rb").read())
        except OSError:
            return None
    return int(kv[key]) if h.hexdigest() == kv.get("sources_sha256") else None


def cpu_baseline(w, budget_s: float = 12.0):
    """The oracle's graft (numpy scatter of payload pages through a block table) timed on
    the host on a bounded sample of the workload's artifact: the first L_s layers."""
    import numpy as np

    from oracle.paging import PagedPool, graft as o_graft
    rng = np.random.default_rng(0)
    n_pages = w.pages_for(w.prefix)
    layers = 4
    payload = rng.integers(0, 65535, size=(layers, 2, n_pages, w.n_kv_heads, w.page_size, w.head_dim),
                           dtype=np.uint16)
    table = rng.permutation(n_pages + 8)[:n_pages]
    pool = PagedPool(layers, n_pages + 8, w.n_kv_heads, w.page_size, w.head_dim, "bf16")
    reps, t = 0, 0.0
    t0 = time.perf_counter()
    while t < budget_s or reps == 0:
        o_graft(pool, payload, table, 0, w.prefix)
        reps += 1
        t = time.perf_counter() - t0
    moved = 2.0 * payload.nbytes * reps
    return {"value": round(moved / t / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"oracle graft of the first {layers} of {w.n_layers} layers of the 4,096-token block "
                      f"({payload.nbytes / 2**20:.0f} MiB payload) x{reps}, {t:.1f} s, single-threaded numpy",
            "per_unit": oracle_attention_units(w)}


def oracle_attention_units(w, rows_sampled: int = 8):
    """The oracle's attention (fp64 numpy) timed per unit on layer 0 of the workload: one
    decode row (the last decode step's, over the whole context) and every 64th suffix row,
    on Gaussian inputs of the workload's shapes and scale (sigma 0.5, drawn with numpy's
    generator: the timing does not depend on the values), best of three calls; extrapolated
    to the step's 512 x 48 prefill row-layers and 64 x 48 decode token-layers.  The products
    go through numpy's BLAS, whose thread count is reported."""
    import numpy as np

    from oracle.attention import attend

    rng = np.random.default_rng(0)
    n_keys = w.ctx_final
    k = rng.standard_normal((n_keys, w.n_kv_heads, w.head_dim)) * 0.5
    v = rng.standard_normal((n_keys, w.n_kv_heads, w.head_dim)) * 0.5
    dec_row = np.array([n_keys - 1])
    suf_rows = w.prefix + np.arange(0, w.suffix, w.suffix // rows_sampled)
    out = {}
    for name, rows in (("decode", dec_row), ("prefill", suf_rows)):
        q = rng.standard_normal((len(rows), w.n_q_heads, w.head_dim)) * 0.5
        best = float("inf")
        for _ in range(3):                      # the first call also pays one-time set-up
            t0 = time.perf_counter()
            attend(q, rows, k, v, w.scale, w.layer_window(0))
            best = min(best, time.perf_counter() - t0)
        out[name] = best / len(rows)
    return {"prefill_row_layer_ms": round(out["prefill"] * 1e3, 3),
            "decode_token_layer_ms": round(out["decode"] * 1e3, 3),
            "step_attention_s_extrapolated": round(
                (w.suffix * out["prefill"] + w.decode_steps * out["decode"]) * w.n_layers, 1),
            "blas_threads": _blas_threads(),
            "sample": f"layer 0: decode row {int(dec_row[0])} over {n_keys} keys, {len(suf_rows)} suffix rows "
                      f"(every {w.suffix // rows_sampled}th), all {w.n_q_heads} heads, single process"}


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max((p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"), default=1)
    except Exception:
        return None


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (this build has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.workload == "12b-store2.85M":
        store_phases(args)
        return
    if args.workload != "12b-block4096":
        workload_phases(args)
        return

    import torch

    from paper_2607_14431_amd import harness as h
    from paper_2607_14431_amd import kvg
    from synth import ROLE_K, ROLE_Q, ROLE_V
    from synth.gpu import raw_chunk
    from synth.workloads import BLOCK12B, SWA12B

    w = BLOCK12B
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    N, S, T = w.prefix, w.suffix, w.decode_steps

    # ---------------------------------------------------------------- setup (untimed)
    fresh = h.new_arm(w, [0], w.ctx_final, seed=100, poison_id=0, spare_pages=11)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    h.fresh_prefix(fresh)                                     # cold prefill of the block
    e1.record(stream)
    torch.cuda.synchronize()
    cold_ms = e0.elapsed_time(e1)
    graft_arm = h.new_arm(w, [0], w.ctx_final, seed=200, poison_id=1, spare_pages=5)
    rp = h.rope_of(w)
    hdr = kvg.kvg_artifact_header_init(fresh.cache, N, 0, rp)
    payload = torch.empty(hdr.payload_bytes, dtype=torch.uint8, device="cuda")
    bt_fresh, bt_graft = fresh.tables[0], graft_arm.tables[0]

    q_s = raw_chunk(w, ROLE_Q, [0], N, S)
    k_s = raw_chunk(w, ROLE_K, [0], N, S)
    v_s = raw_chunk(w, ROLE_V, [0], N, S)
    dec_in = [(raw_chunk(w, ROLE_Q, [0], N + S + i, 1), raw_chunk(w, ROLE_K, [0], N + S + i, 1),
               raw_chunk(w, ROLE_V, [0], N + S + i, 1)) for i in range(T)]
    meta_s = graft_arm.meta(N)
    meta_d = [graft_arm.meta(N + S + i) for i in range(T)]
    ws = torch.empty(kvg.kvg_prefill_workspace_bytes(graft_arm.cache, meta_s, w.n_layers, S), dtype=torch.uint8,
                     device="cuda")
    ws_dec = kvg.decode_workspace(graft_arm.cache, meta_d[-1], w.n_layers)
    out_s = torch.empty((w.n_layers, 1, S, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    out_d = torch.empty((T, w.n_layers, 1, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")

    phases = ["deposit", "graft", "prefill", "decode"]
    ev = {p: [] for p in phases}
    dec_ev = []                                   # one event pair per decode launch

    def step(record: bool):
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(5)] if record else None
        if record:
            marks[0].record(stream)
        kvg.kvg_deposit(fresh.cache, bt_fresh, 0, N, payload, stream)
        if record:
            marks[1].record(stream)
        kvg.kvg_graft(graft_arm.cache, hdr, payload, bt_graft, 0, 0, 0, stream)
        if record:
            marks[2].record(stream)
        kvg.kvg_prefill_attn(graft_arm.cache, meta_s, rp, 0, w.n_layers, S, q_s, k_s, v_s, w.scale, out_s, ws,
                             stream)
        if record:
            marks[3].record(stream)
        for i in range(T):
            q, k, v = dec_in[i]
            if record:
                d0, d1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                d0.record(stream)
            kvg.kvg_decode_attn(graft_arm.cache, meta_d[i], rp, 0, w.n_layers, q, k, v, w.scale, out_d[i], ws_dec,
                                stream)
            if record:
                d1.record(stream)
                dec_ev.append((i, d0, d1))
        if record:
            marks[4].record(stream)
            for j, p in enumerate(phases):
                ev[p].append((marks[j], marks[j + 1]))

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    ph = {p: sum(a.elapsed_time(b) for a, b in ev[p]) / args.steps for p in phases}
    dec_launch_ms = [(i, a.elapsed_time(b)) for i, a, b in dec_ev]

    # ---------------------------------------------------------------- verification (untimed)
    verdict = None
    res_fresh = res_graft = None
    if not args.no_verify:
        res_graft = (out_s.clone(), out_d.clone())
        _, restored = h.deposit(graft_arm, 0, 0, N, 0)
        res_fresh = h.continue_arm(fresh)
        torch.cuda.synchronize()
        sha = lambda t: hashlib.sha256(t.contiguous().view(torch.uint8).cpu().numpy().tobytes()).hexdigest()  # noqa
        verdict = (sha(payload) == sha(restored) and h.bytes_equal(res_fresh.suffix, res_graft[0])
                   and h.bytes_equal(res_fresh.decode, res_graft[1]))

    # ---------------------------------------------------------------- figures
    pay = float(hdr.payload_bytes)
    graft_bytes = 2.0 * pay                                   # payload read + pool written
    graft_gbps = graft_bytes / (ph["graft"] * 1e-3) / 1e9
    deposit_gbps = graft_bytes / (ph["deposit"] * 1e-3) / 1e9
    dec_bytes_launch = sum(decode_launch_bytes(w, N + S + i) for i in range(T)) / T
    dec_launch_avg_ms = sum(ms for _, ms in dec_launch_ms) / len(dec_launch_ms)
    dec_gbps = dec_bytes_launch / (dec_launch_avg_ms * 1e-3) / 1e9
    decode_tok_s = w.batch * T / (ph["decode"] * 1e-3)
    decode_frac = dec_gbps / HBM_PEAK_GBPS
    prefill_flop = prefill_flops(w, N, S)
    prefill_tflops = prefill_flop / (ph["prefill"] * 1e-3) / 1e12

    extras = {}
    if not args.no_extras:
        extras.update(digest_figures(kvg, torch, stream, w, payload, int(hdr.payload_bytes)))
        launches = dict(rp=rp, meta_s=meta_s, q_s=q_s, k_s=k_s, v_s=v_s, ws=ws, out_s=out_s, meta_d=meta_d,
                        dec_in=dec_in, ws_dec=ws_dec, out_d=out_d)
        extras.update(window_figures(kvg, torch, stream, w, graft_arm.cache, launches, SWA12B.layer_windows))
        extras.update(per_layer_figures(kvg, torch, stream, w, graft_arm.cache, launches))
        extras.update(logit_figures(h, kvg, torch, stream, w, res_fresh, res_graft))
        extras.update(fp8_figures(h, kvg, torch, stream, w))
        extras.update(relocation_figures(h, kvg, torch, stream, w, hdr, payload))

    line = {
        "metric": "graft restore GB/s; decode-attn tok/s over grafted ctx (% HBM peak); graft==fresh",
        "value": round(graft_gbps, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "n_layers": w.n_layers, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "block_tokens": N, "suffix": S, "decode_steps": T, "batch": w.batch,
                   "page_size": w.page_size},
        "graft_eq_fresh": verdict,
        "decode_tok_s": round(decode_tok_s, 1),
        "decode_hbm_frac": round(decode_frac, 4),
        "decode_ms_per_step": round(ph["decode"] / T, 4),
        "deposit_GBps": round(deposit_gbps, 1),
        "prefill_TFLOPs": round(prefill_tflops, 2),
        "phases_ms": {p: round(v, 4) for p, v in ph.items()},
        "cold_prefill_ms": round(cold_ms, 2),
        "roofline": {"kernel": "kvg_decode_attn: decode_kernel<bf16, 256, 2> + decode_merge_kernel",
                     "bound": "hbm", "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(decode_frac, 4), "traffic": measured_traffic("decode_bytes_per_launch"),
                     "bytes_per_launch": round(dec_bytes_launch), "avg_launch_us": round(dec_launch_avg_ms * 1e3, 2)},
        "rooflines_other": {
            "graft_kernel": {"bound": "hbm", "achieved": round(graft_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                             "frac": round(graft_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": graft_bytes},
            "deposit_kernel": {"bound": "hbm", "achieved": round(deposit_gbps, 1), "peak": HBM_PEAK_GBPS,
                               "unit": "GB/s", "frac": round(deposit_gbps / HBM_PEAK_GBPS, 4),
                               "bytes_per_launch": graft_bytes},
            "prefill (append + prefill_mfma_kernel)": {
                "bound": "mfma", "achieved": round(prefill_tflops, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(prefill_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                "flop_per_launch": prefill_flop},
            **extras,
        },
    }
    copy_gbps = measured_copy_gbps(torch, stream)
    line["runtime_copy_GBps"] = round(copy_gbps, 1)             # hipMemcpy-class D2D copy of 1 GiB
    line["roofline"]["frac_of_runtime_copy"] = round(dec_gbps / copy_gbps, 4)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(line), flush=True)


def measured_copy_gbps(torch, stream) -> float:
    """Rate of the runtime's own 1 GiB device-to-device copy on this GPU (bytes read +
    written per second): the device-copy reference the HBM-bound kernels are also compared
    with (this library's copy kernels stream faster than it)."""
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    ms = []
    for rep in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        dst.copy_(src)
        e1.record(stream)
        torch.cuda.synchronize()
        if rep:
            ms.append(e0.elapsed_time(e1))
    return 2.0 * n / (sum(ms) / len(ms) * 1e-3) / 1e9


def workload_phases(args):
    """Full-size 12b-window32k (16 sequences, 8 store blocks of 4,096 each grafted at its own
    position) or 31b-reloc16k (8 sequences, a 16,384-token block each, grafted 8,192
    positions away from where it was captured): every graft, the suffix prefill of all
    sequences and the decode steps, each timed with events on the launch stream."""
    import gc

    import torch

    from paper_2607_14431_amd import harness as h
    from paper_2607_14431_amd import kvg
    from synth.workloads import RELOC31B, WINDOW12B, scaled

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    graft_ms, graft_bytes = [], 0.0
    if args.workload == "12b-window32k":
        w = WINDOW12B
        seqs = list(range(w.batch))
        g = h.new_arm(w, seqs, w.ctx_final, seed=300, poison_id=1)
        for bi, s in enumerate(seqs):
            for j in range(w.blocks_per_seq):
                hdr, payload = h.store_artifact(w, w.seq_block(s, j), j)
                e0, e1 = ev(), ev()
                e0.record(stream)
                h.graft(g, bi, hdr, payload, j * w.block_tokens, j * w.block_tokens)
                e1.record(stream)
                torch.cuda.synchronize()
                graft_ms.append(e0.elapsed_time(e1))
                graft_bytes += 2.0 * hdr.payload_bytes
                del payload
        relocated = False
    else:
        w0 = scaled(RELOC31B, start_pos=0)
        w = RELOC31B
        seqs = list(range(w.batch))
        fresh = h.new_arm(w0, seqs, w0.ctx_final, seed=400, poison_id=0)
        h.fresh_prefix(fresh, append_only=True, chunk=4096)
        arts = [h.deposit(fresh, bi, 0, w0.prefix, 0) for bi in range(len(seqs))]
        del fresh
        gc.collect()
        torch.cuda.empty_cache()
        g = h.new_arm(w, seqs, w.ctx_final, seed=402, poison_id=1)
        for bi, (hdr, payload) in enumerate(arts):
            e0, e1 = ev(), ev()
            e0.record(stream)
            h.graft(g, bi, hdr, payload, 0, w.start_pos, relocate=True)
            e1.record(stream)
            torch.cuda.synchronize()
            graft_ms.append(e0.elapsed_time(e1))
            graft_bytes += 2.0 * hdr.payload_bytes
        del arts
        gc.collect()
        torch.cuda.empty_cache()
        relocated = True
    # the first graft pays one-time costs (first touch of pages): it is left out
    t_graft = sum(graft_ms[1:]) / (len(graft_ms) - 1)
    per_graft = graft_bytes / len(graft_ms)
    graft_gbps = per_graft / (t_graft * 1e-3) / 1e9

    N, S, T, B = w.prefix, w.suffix, w.decode_steps, w.batch
    from synth import ROLE_K, ROLE_Q, ROLE_V
    from synth.gpu import raw_chunk
    rp = h.rope_of(w)
    # suffix prefill of every sequence: inputs and buffers first, a warm-up call (it rewrites
    # the same K/V bytes), then the timed call
    q_s, k_s, v_s = (raw_chunk(w, r, seqs, N, S) for r in (ROLE_Q, ROLE_K, ROLE_V))
    meta_s = g.meta(N)
    ws_s = torch.empty(kvg.kvg_prefill_workspace_bytes(g.cache, meta_s, w.n_layers, S), dtype=torch.uint8,
                       device="cuda")
    out_s = torch.empty((w.n_layers, B, S, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    pf_ms = []
    for rep in range(2):
        e0, e1 = ev(), ev()
        e0.record(stream)
        kvg.kvg_prefill_attn(g.cache, meta_s, rp, 0, w.n_layers, S, q_s, k_s, v_s, w.scale, out_s, ws_s, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        pf_ms.append(e0.elapsed_time(e1))
    t_prefill = pf_ms[-1]
    del q_s, k_s, v_s, ws_s, out_s
    prefill_flop = B * prefill_flops(w, N, S)
    dec_ms = []
    ws = kvg.decode_workspace(g.cache, g.meta(N + S + T - 1), w.n_layers)
    out = torch.empty((w.n_layers, B, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    for i in range(T):
        t0 = N + S + i
        q, k, v = (raw_chunk(w, r, seqs, t0, 1)[:, :, 0].contiguous() for r in (ROLE_Q, ROLE_K, ROLE_V))
        meta = g.meta(t0)
        e0, e1 = ev(), ev()
        e0.record(stream)
        kvg.kvg_decode_attn(g.cache, meta, rp, 0, w.n_layers, q, k, v, w.scale, out, ws, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        dec_ms.append(e0.elapsed_time(e1))
    t_dec = sum(dec_ms) / T
    dec_bytes = B * sum(decode_launch_bytes(w, N + S + i) for i in range(T)) / T
    dec_gbps = dec_bytes / (t_dec * 1e-3) / 1e9
    line = {
        "metric": "graft restore GB/s; decode-attn tok/s over grafted ctx (% HBM peak)",
        "value": round(graft_gbps, 1), "unit": "GB/s", "n_gpus": 1, "higher_is_better": True,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "n_layers": w.n_layers, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "prefix": N, "suffix": S, "decode_steps": T, "batch": B,
                   "relocated_by": w.start_pos - w.own_pos if relocated else 0},
        "graft": {"bound": "hbm", "achieved": round(graft_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                  "frac": round(graft_gbps / HBM_PEAK_GBPS, 4), "grafts": len(graft_ms),
                  "bytes_per_graft": per_graft, "ms_per_graft": round(t_graft, 4)},
        "prefill": {"bound": "mfma", "achieved": round(prefill_flop / (t_prefill * 1e-3) / 1e12, 1),
                    "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(prefill_flop / (t_prefill * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                    "flop": prefill_flop, "ms": round(t_prefill, 3)},
        "decode": {"bound": "hbm", "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                   "frac": round(dec_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": round(dec_bytes),
                   "ms_per_step": round(t_dec, 3), "tok_s": round(B / (t_dec * 1e-3), 1)},
        "runtime_copy_GBps": round(measured_copy_gbps(torch, stream), 1),
    }
    print(json.dumps(line), flush=True)


STORE_DEPTH_BLOCKS = (0, 81, 169, 344, 520, 607, 688, 696)   # the paper's needle depths + the partial last block


def store_phases(args):
    """The 2,854,766-token store (697 blocks of 4,096, the last partial) paged through a
    32,768-token window of 8 direct-mapped slots shared by 32 decoding sequences.  Per access
    of block b (at the paper's needle depths): graft from host-pinned memory into slot
    b mod 8 at its own position, a 35-token suffix prefill for every sequence, 8 decode
    steps; each timed with events on the launch stream.  The block's on-host form (a fresh
    computation and deposit) and the access's inputs are produced before it, untimed.  The
    metric is the access latency against depth; the graft rate is PCIe-bound (host memory
    read by the kernel) and is never an HBM figure."""
    import torch

    from paper_2607_14431_amd import harness as h
    from synth.workloads import STORE12B

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    w = STORE12B
    win = h.StoreWindow(w)
    pinned = h.PinnedPayload(h.kvg.kvg_payload_bytes(win.cache, w.block_tokens))
    for b in range(win.slots):                      # initial window fill (untimed)
        win.graft(b, win.materialize(b, pinned), pinned)
    torch.cuda.synchronize()
    from synth import ROLE_K, ROLE_Q, ROLE_V
    from synth.gpu import raw_chunk
    kvg = h.kvg
    arm, N, S, T = win.arm, win.win_tokens, w.suffix, w.decode_steps
    rows = []
    for b in STORE_DEPTH_BLOCKS:
        hdr = win.materialize(b, pinned)
        # inputs, buffers and workspaces of the access, made before the timed region
        vw = win.view()
        arm.w = vw
        q_s, k_s, v_s = (raw_chunk(vw, r, arm.seqs, N, S) for r in (ROLE_Q, ROLE_K, ROLE_V))
        meta_s = arm.meta(N)
        ws_s = torch.empty(kvg.kvg_prefill_workspace_bytes(arm.cache, meta_s, w.n_layers, S), dtype=torch.uint8,
                           device="cuda")
        out_s = torch.empty((w.n_layers, win.batch, S, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
        dec = [tuple(raw_chunk(vw, r, arm.seqs, N + S + i, 1) for r in (ROLE_Q, ROLE_K, ROLE_V)) + (arm.meta(N + S + i),)
               for i in range(T)]
        ws_d = kvg.decode_workspace(arm.cache, arm.meta(N + S + T - 1), w.n_layers)
        out_d = torch.empty((T, w.n_layers, win.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
        rp = h.rope_of(vw)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        win.graft(b, hdr, pinned)
        ev[1].record(stream)
        kvg.kvg_prefill_attn(arm.cache, meta_s, rp, 0, w.n_layers, S, q_s, k_s, v_s, vw.scale, out_s, ws_s)
        ev[2].record(stream)
        for i, (q, k, v, meta) in enumerate(dec):
            kvg.kvg_decode_attn(arm.cache, meta, rp, 0, w.n_layers, q, k, v, vw.scale, out_d[i], ws_d)
        ev[3].record(stream)
        torch.cuda.synchronize()
        t = [ev[i].elapsed_time(ev[i + 1]) for i in range(3)]
        rows.append({"block": b, "depth_tokens": b * w.block_tokens, "block_tokens": int(hdr.n_tokens),
                     "graft_ms": round(t[0], 3), "graft_GBps_pcie": round(hdr.payload_bytes / (t[0] * 1e-3) / 1e9, 1),
                     "suffix_prefill_ms": round(t[1], 3), "decode_ms": round(t[2], 3),
                     "access_ms": round(sum(t), 3)})
        print(f"access block {b}: {rows[-1]}", file=sys.stderr, flush=True)
    full = [r for r in rows if r["block_tokens"] == w.block_tokens]
    mean_access = sum(r["access_ms"] for r in full) / len(full)
    line = {
        "metric": "store access latency vs depth (graft from host + suffix prefill + decode)",
        "value": round(mean_access, 3), "unit": "ms per access", "n_gpus": 1, "higher_is_better": False,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": "12b-store2.85M", "store_tokens": w.store_tokens, "store_blocks": w.store_blocks,
                   "window_slots": win.slots, "batch": win.batch, "suffix": w.suffix, "decode_steps": w.decode_steps},
        "max_over_min_graft_ms": round(max(r["graft_ms"] for r in full) / min(r["graft_ms"] for r in full), 3),
        "depths": rows,
    }
    print(json.dumps(line), flush=True)


def visible(n_keys: int, window: int) -> int:
    """Keys a query sees when its causal prefix holds n_keys keys: all of them, or the last
    `window` for a windowed layer (keys i - W < j <= i)."""
    return n_keys if window == 0 else min(n_keys, window)


def decode_launch_bytes(w, ctx: int, windows=None) -> float:
    """Algorithmic HBM bytes of one decode launch over ctx cached tokens: the visible cached
    K/V read (every layer, or the last W - 1 keys before the new token for a windowed
    layer), the raw q/k/v read, the new token's K/V written, the fp32 outputs written."""
    kv_layer = 2 * w.n_kv_heads * w.head_dim * w.elem_bytes
    windows = windows or (0,) * w.n_layers
    cached = sum(kv_layer * (visible(ctx + 1, W) - 1) for W in windows)
    raw_bytes = 4 if w.raw_dtype == "f32" else 2                 # an fp8 cache takes bf16 inputs
    row_in = (w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim * raw_bytes * w.n_layers
    row_out = w.n_q_heads * w.head_dim * 4 * w.n_layers
    return cached + row_in + kv_layer * w.n_layers + row_out


def prefill_flops(w, ctx: int, rows: int, windows=None) -> float:
    """Algorithmic flops of a prefill of `rows` rows over ctx cached tokens: 4 Hq D per
    (row, visible key) pair (QK^T and PV, multiply-add = 2 flops), every layer."""
    windows = windows or (0,) * w.n_layers
    return 4.0 * w.n_q_heads * w.head_dim * sum(visible(ctx + i + 1, W) for W in windows for i in range(rows))


def digest_figures(kvg, torch, stream, w, payload, payload_bytes: int) -> dict:
    """SHA-256 of every (layer, K/V, page, head) slab of the artifact, the Merkle root over
    them and the dedup map (not part of the step), timed with events on the launch stream."""
    slab = w.page_size * w.head_dim * w.elem_bytes
    n_leaves = payload_bytes // slab
    digests = torch.empty((n_leaves, 32), dtype=torch.uint8, device="cuda")
    root = torch.zeros(32, dtype=torch.uint8, device="cuda")
    mws = torch.empty(kvg.kvg_merkle_workspace_bytes(n_leaves), dtype=torch.uint8, device="cuda")
    first_idx = torch.empty(n_leaves, dtype=torch.int64, device="cuda")
    n_unres = torch.zeros(1, dtype=torch.int32, device="cuda")
    dws = torch.empty(kvg.kvg_dedup_workspace_bytes(n_leaves), dtype=torch.uint8, device="cuda")
    dig_ms = {"leaf_digests": [], "merkle_root": [], "dedup_map": []}
    for rep in range(4):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record(stream)
        kvg.kvg_leaf_digests(payload, slab, digests, stream=stream)
        e[1].record(stream)
        kvg.kvg_merkle_root(digests, n_leaves, root, mws, stream=stream)
        e[2].record(stream)
        kvg.kvg_dedup_map(digests, n_leaves, first_idx, n_unres, dws, stream=stream)
        e[3].record(stream)
        torch.cuda.synchronize()
        if rep:                                   # the first pass is a warm-up
            for j, k in enumerate(dig_ms):
                dig_ms[k].append(e[j].elapsed_time(e[j + 1]))
    avg = {k: sum(v) / len(v) for k, v in dig_ms.items()}
    n_blocks = n_leaves * (slab // 64 + 1)        # data blocks plus each leaf's padding block
    sha_gops = n_blocks * SHA256_OPS_PER_BLOCK / (avg["leaf_digests"] * 1e-3) / 1e9
    return {"leaf_digests (SHA-256 of 8 KiB slabs of the artifact, not in the step)": {
        "bound": "alu", "achieved": round(sha_gops, 1), "peak": VALU_PEAK_GOPS, "unit": "Gop/s",
        "frac": round(sha_gops / VALU_PEAK_GOPS, 4), "ops_per_launch": n_blocks * SHA256_OPS_PER_BLOCK,
        "GBps": round(payload_bytes / (avg["leaf_digests"] * 1e-3) / 1e9, 1), "ms": round(avg["leaf_digests"], 4),
        "merkle_root_ms": round(avg["merkle_root"], 4), "dedup_map_ms": round(avg["dedup_map"], 4),
        "leaves": n_leaves, "dedup_unresolved": int(n_unres.item())}}


def logit_figures(h, kvg, torch, stream, w, res_fresh, res_graft) -> dict:
    """The synthetic soft-capped head (262,144 x 4,096 bf16) over the last layer's outputs (not
    part of the step): its launch time for one row (a decode step, W streamed once) and for
    the 50 sample rows, and, when the arms were kept, the logit-level verdict over 50 rows
    spread across the suffix and the decode steps: SHA-256 of each row, KL, argmax."""
    wt = h.head_weights(w)
    V, H = wt.vocab, wt.hidden
    out = {}
    for rows in (1, 50):
        hid = torch.randn((rows, H), dtype=torch.float32, device="cuda") * 0.02
        lg = torch.empty((rows, V), dtype=torch.float32, device="cuda")
        ws = torch.empty(kvg.kvg_logits_workspace_bytes(rows, H), dtype=torch.uint8, device="cuda")
        ms = []
        for rep in range(6):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            kvg.kvg_logits(hid, wt.packed, V, h.HEAD_CAP, lg, ws, stream)
            e1.record(stream)
            torch.cuda.synchronize()
            if rep:
                ms.append(e0.elapsed_time(e1))
        t = sum(ms) / len(ms)
        byts = V * H * 2 + rows * H * 4 + rows * V * 4    # algorithmic: W once (the kernel reads
                                                            # it once per 32 rows)
        gbps = byts / (t * 1e-3) / 1e9
        out[f"logit head, {rows} row{'s' if rows > 1 else ''} x {V:,} x {H:,} bf16 (not in the step)"] = {
            "bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": byts, "avg_launch_us": round(t * 1e3, 2)}
    if res_fresh is not None:
        n_rows = w.suffix + w.decode_steps
        pick = sorted({round(i * (n_rows - 1) / 49) for i in range(50)})
        graft = h.ArmResult(res_graft[0], res_graft[1])
        lf = h.logits(h.hidden_rows(res_fresh, 0, pick), wt)
        lgr = h.logits(h.hidden_rows(graft, 0, pick), wt)
        out["logit verdict, graft vs fresh (Eq. 1-2)"] = h.exactness_stats(lgr, lf)
    return out


def relocation_figures(h, kvg, torch, stream, w, hdr, payload) -> dict:
    """The block grafted 8,192 positions away from where it was captured (not part of the
    step): keys re-rotated by the offset (graft_relocate_k_kernel), values copied
    (graft_kernel), into a scratch cache.  Algorithmic bytes: the payload read and the pages
    written, as for the own-position graft."""
    arm = h.new_arm(w, [0], w.ctx_final, seed=230, poison_id=1, start_pos=8192)
    ms = []
    for rep in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        kvg.kvg_graft(arm.cache, hdr, payload, arm.tables[0], 0, 8192, kvg.KVG_GRAFT_ALLOW_RELOCATE, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        if rep:                                   # the first pass is a warm-up
            ms.append(e0.elapsed_time(e1))
    t = sum(ms) / len(ms)
    byts = 2.0 * hdr.payload_bytes
    return {"relocated graft, +8,192 positions (graft_relocate_k_kernel + graft_kernel, not in the step)": {
        "bound": "hbm", "achieved": round(byts / (t * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
        "frac": round(byts / (t * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4), "bytes_per_launch": byts, "ms": round(t, 4)}}


def fp8_figures(h, kvg, torch, stream, w) -> dict:
    """The same block with an fp8 E4M3 cache (not part of the step): bf16 inputs rounded once
    when stored, so the payload is half the bytes.  Deposit and graft of the block, the
    suffix prefill and the 64 decode steps, timed with events on the launch stream."""
    import dataclasses
    from synth import ROLE_K, ROLE_Q, ROLE_V
    from synth.gpu import raw_chunk
    w8 = dataclasses.replace(w, dtype="fp8")
    N, S, T = w8.prefix, w8.suffix, w8.decode_steps
    fresh = h.new_arm(w8, [0], w8.ctx_final, seed=120, poison_id=0, spare_pages=11)
    h.fresh_prefix(fresh, append_only=True)
    g = h.new_arm(w8, [0], w8.ctx_final, seed=220, poison_id=1, spare_pages=5)
    rp = h.rope_of(w8)
    hdr = kvg.kvg_artifact_header_init(fresh.cache, N, 0, rp)
    payload = torch.empty(hdr.payload_bytes, dtype=torch.uint8, device="cuda")
    q_s, k_s, v_s = (raw_chunk(w8, r, [0], N, S) for r in (ROLE_Q, ROLE_K, ROLE_V))
    meta_s = g.meta(N)
    ws = torch.empty(kvg.kvg_prefill_workspace_bytes(g.cache, meta_s, w8.n_layers, S), dtype=torch.uint8,
                     device="cuda")
    out_s = torch.empty((w8.n_layers, 1, S, w8.n_q_heads, w8.head_dim), dtype=torch.float32, device="cuda")
    dec_in = [tuple(raw_chunk(w8, r, [0], N + S + i, 1) for r in (ROLE_Q, ROLE_K, ROLE_V)) for i in range(T)]
    meta_d = [g.meta(N + S + i) for i in range(T)]
    ws_d = kvg.decode_workspace(g.cache, meta_d[-1], w8.n_layers)
    out_d = torch.empty((w8.n_layers, 1, w8.n_q_heads, w8.head_dim), dtype=torch.float32, device="cuda")
    ms = {"deposit": [], "graft": [], "prefill": [], "decode": []}
    for rep in range(3):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4 + 2 * T)]
        e[0].record(stream)
        kvg.kvg_deposit(fresh.cache, fresh.tables[0], 0, N, payload, stream)
        e[1].record(stream)
        kvg.kvg_graft(g.cache, hdr, payload, g.tables[0], 0, 0, 0, stream)
        e[2].record(stream)
        kvg.kvg_prefill_attn(g.cache, meta_s, rp, 0, w8.n_layers, S, q_s, k_s, v_s, w8.scale, out_s, ws, stream)
        e[3].record(stream)
        for i in range(T):
            q, k, v = dec_in[i]
            e[4 + 2 * i].record(stream)
            kvg.kvg_decode_attn(g.cache, meta_d[i], rp, 0, w8.n_layers, q, k, v, w8.scale, out_d, ws_d, stream)
            e[5 + 2 * i].record(stream)
        torch.cuda.synchronize()
        if rep:                                   # the first pass is a warm-up
            for j, k in enumerate(("deposit", "graft", "prefill")):
                ms[k].append(e[j].elapsed_time(e[j + 1]))
            ms["decode"] += [e[4 + 2 * i].elapsed_time(e[5 + 2 * i]) for i in range(T)]
    avg = {k: sum(v) / len(v) for k, v in ms.items()}
    pay = 2.0 * hdr.payload_bytes
    dec_bytes = sum(decode_launch_bytes(w8, N + S + i) for i in range(T)) / T
    dec_gbps = dec_bytes / (avg["decode"] * 1e-3) / 1e9
    pf_flop = prefill_flops(w8, N, S)
    out = {"fp8 E4M3 cache: graft_kernel (not in the step)": {
               "bound": "hbm", "achieved": round(pay / (avg["graft"] * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBPS,
               "unit": "GB/s", "frac": round(pay / (avg["graft"] * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
               "bytes_per_launch": pay, "ms": round(avg["graft"], 4), "deposit_ms": round(avg["deposit"], 4)},
           "fp8 E4M3 cache: decode_kernel + decode_merge_kernel (not in the step)": {
               "bound": "hbm", "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
               "frac": round(dec_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": round(dec_bytes),
               "avg_launch_us": round(avg["decode"] * 1e3, 2), "tok_s": round(w8.batch / (avg["decode"] * 1e-3), 1)},
           "fp8 E4M3 cache: suffix prefill, append + prefill_mfma_kernel<fp8> (not in the step)": {
               "bound": "mfma", "achieved": round(pf_flop / (avg["prefill"] * 1e-3) / 1e12, 1),
               "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
               "frac": round(pf_flop / (avg["prefill"] * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
               "flop_per_launch": pf_flop, "ms": round(avg["prefill"], 3)}}
    return out


def window_figures(kvg, torch, stream, w, cache, x: dict, windows) -> dict:
    """The grafted cache read by a model whose layers attend to sliding windows (not part of
    the step): the suffix prefill and the decode steps again, with per-layer windows; the
    launches rewrite the same K/V bytes."""
    import dataclasses
    swa_cache = dataclasses.replace(cache, windows=tuple(windows))
    N, S, T = w.prefix, w.suffix, w.decode_steps
    ms = {"prefill": [], "decode": []}
    for rep in range(3):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2 + 2 * T)]
        e[0].record(stream)
        kvg.kvg_prefill_attn(swa_cache, x["meta_s"], x["rp"], 0, w.n_layers, S, x["q_s"], x["k_s"], x["v_s"],
                             w.scale, x["out_s"], x["ws"], stream)
        e[1].record(stream)
        for i in range(T):
            q, k, v = x["dec_in"][i]
            e[2 + 2 * i].record(stream)
            kvg.kvg_decode_attn(swa_cache, x["meta_d"][i], x["rp"], 0, w.n_layers, q, k, v, w.scale, x["out_d"][i],
                                x["ws_dec"], stream)
            e[3 + 2 * i].record(stream)
        torch.cuda.synchronize()
        if rep:                                   # the first pass is a warm-up
            ms["prefill"].append(e[0].elapsed_time(e[1]))
            ms["decode"] += [e[2 + 2 * i].elapsed_time(e[3 + 2 * i]) for i in range(T)]
    avg = {k: sum(v) / len(v) for k, v in ms.items()}
    dec_bytes = sum(decode_launch_bytes(w, N + S + i, windows) for i in range(T)) / T
    dec_gbps = dec_bytes / (avg["decode"] * 1e-3) / 1e9
    pf_flop = prefill_flops(w, N, S, windows)
    pf_tflops = pf_flop / (avg["prefill"] * 1e-3) / 1e12
    n_win = sum(1 for W in windows if W)
    desc = f"{max(windows):,}-key windows on {n_win} of {len(windows)} layers, not in the step"
    return {
        f"decode ({desc})": {
            "bound": "hbm", "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(dec_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": round(dec_bytes),
            "avg_launch_us": round(avg["decode"] * 1e3, 2), "tok_s": round(w.batch / (avg["decode"] * 1e-3), 1)},
        f"prefill ({desc})": {
            "bound": "mfma", "achieved": round(pf_tflops, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(pf_tflops / MFMA_BF16_PEAK_TFLOPS, 4), "flop_per_launch": pf_flop,
            "ms": round(avg["prefill"], 4)},
    }


def per_layer_figures(kvg, torch, stream, w, cache, x: dict) -> dict:
    """The step's suffix prefill and first decode step launched one layer at a time (48
    launches each, not part of the step) against the all-layer launches the step makes: a
    single layer's decode reads only 1/48 of the bytes (38 MB), too little to fill the GPU."""
    N, S, L = w.prefix, w.suffix, w.n_layers
    q, k, v = x["dec_in"][0]
    ms = {"prefill": [], "decode": []}
    for rep in range(3):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record(stream)
        for l in range(L):
            kvg.kvg_prefill_attn(cache, x["meta_s"], x["rp"], l, 1, S, x["q_s"][l:l + 1], x["k_s"][l:l + 1],
                                 x["v_s"][l:l + 1], w.scale, x["out_s"][l:l + 1], x["ws"], stream)
        e[1].record(stream)
        e[2].record(stream)
        for l in range(L):
            kvg.kvg_decode_attn(cache, x["meta_d"][0], x["rp"], l, 1, q[l:l + 1], k[l:l + 1], v[l:l + 1], w.scale,
                                x["out_d"][0][l:l + 1], x["ws_dec"], stream)
        e[3].record(stream)
        torch.cuda.synchronize()
        if rep:                                   # the first pass is a warm-up
            ms["prefill"].append(e[0].elapsed_time(e[1]))
            ms["decode"].append(e[2].elapsed_time(e[3]))
    avg = {k_: sum(v_) / len(v_) for k_, v_ in ms.items()}
    dec_bytes = decode_launch_bytes(w, N + S)
    dec_gbps = dec_bytes / (avg["decode"] * 1e-3) / 1e9
    pf_flop = prefill_flops(w, N, S)
    pf_tflops = pf_flop / (avg["prefill"] * 1e-3) / 1e12
    return {
        f"decode, {L} one-layer launches (not in the step)": {
            "bound": "hbm", "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(dec_gbps / HBM_PEAK_GBPS, 4), "bytes_per_call": round(dec_bytes),
            "us_per_layer_launch": round(avg["decode"] * 1e3 / L, 2), "us_all_layers": round(avg["decode"] * 1e3, 2)},
        f"prefill, {L} one-layer launches (not in the step)": {
            "bound": "mfma", "achieved": round(pf_tflops, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(pf_tflops / MFMA_BF16_PEAK_TFLOPS, 4), "flop_per_call": pf_flop,
            "us_per_layer_launch": round(avg["prefill"] * 1e3 / L, 2), "ms_all_layers": round(avg["prefill"], 4)},
    }


if __name__ == "__main__":
    main()
