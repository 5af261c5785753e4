"""Benchmark of the byte-exact KV grafting hot path on one MI355X.

One step = the whole hot path over one batch of synthetic input, all inputs already
resident in HBM.  The headline workload is the 12B-class 32k window (48 layers, 16 query /
8 KV heads, head_dim 256, bf16, page size 16): 16 sequences, each with its own block table
and a 32,768-token window filled by 8 blocks of 4,096 tokens drawn from a seeded 256-block
store (block j of a window sits at its own position 4,096 j), a 512-token suffix and 64
decode steps.  A step deposits every block of the batch (128 x 1.5 GiB gathers) and grafts
it back at its own position through a ring of payload buffers (128 scatters), prefills the
16 suffixes over their grafted windows, then runs the 64 decode steps of the batch.

Prints one JSON line.  `value` is the graft restore rate (payload bytes read + pool bytes
written, per graft launch time).  Beside it: decode tokens/s and its HBM fraction, the
graft==fresh verdict (a sequence recomputed fresh at batch 1, byte-compared, outside the
timed region), per-phase times, the roofline of the dominant kernel (the decode call), the
other configurations (12B single block with its extras, 31B block relocated by +8,192, the
2.85M-token store paged through a shared window, the tiny fp32 case), and the oracle's CPU
baseline on the host's cores.
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
PAYLOAD_RING = 8                # payload buffers the 32k-window step cycles its 128 blocks through

WORKLOADS = ["all", "12b-window32k", "12b-block4096", "31b-reloc16k", "12b-store2.85M"]


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-verify", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the figures taken after the timed steps (other configurations, content "
                        "digests, sliding-window launches), so that a counter pass sees only the step's kernels")
    p.add_argument("--workload", default="all", choices=WORKLOADS,
                   help="all (default): the 32k-window step as the headline with the other configurations "
                        "beside it; a single name runs that configuration alone")
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


def measured_traffic(profile: str, key: str):
    """HBM bytes per launch of a kernel as counted by rocprofv3 (FETCH_SIZE + WRITE_SIZE,
    scaled by a plain copy's counts) in a committed traffic summary under profiles/, or None
    when the summary is absent or the kernel's sources have changed since the counters were
    taken."""
    try:
        text = open(os.path.join(ROOT, "profiles", profile)).read()
    except OSError:
        return None
    # "k = v" lines; each figure belongs to the nearest "sources" / "sources_sha256" above it
    sources = digest = None
    for ln in text.splitlines():
        if " = " not in ln:
            continue
        k, v = ln.strip().split(" = ", 1)
        if k == "sources":
            sources, digest = v.split(), None
        elif k == "sources_sha256":
            digest = v
        elif k == key:
            if not sources or not digest:
                return None
            h = hashlib.sha256()
            for rel in sources:
                try:
                    h.update(open(os.path.join(ROOT, rel), "rb").read())
                except OSError:
                    return None
            return int(v) if h.hexdigest() == digest else None
    return None


# ------------------------------------------------------------------------------ CPU baseline
def host_info() -> dict:
    """The host the CPU baseline runs on: usable cores, CPU model, last-level cache."""
    import platform
    cores = len(os.sched_getaffinity(0))
    model = platform.processor() or ""
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    # last-level cache reachable from the usable cores: the sum over the distinct highest-level
    # cache instances they sit on (one per core complex on parts with several)
    seen, llc = set(), 0
    for cpu in sorted(os.sched_getaffinity(0)):
        base = f"/sys/devices/system/cpu/cpu{cpu}/cache"
        try:
            idxs = [i for i in os.listdir(base) if i.startswith("index")]
            top = max(idxs, key=lambda i: int(open(f"{base}/{i}/level").read()))
            shared = open(f"{base}/{top}/shared_cpu_list").read().strip()
            size = open(f"{base}/{top}/size").read().strip()
        except (OSError, ValueError):
            continue
        if shared in seen:
            continue
        seen.add(shared)
        mult = {"K": 1 << 10, "M": 1 << 20, "G": 1 << 30}.get(size[-1], 1)
        llc += int(size[:-1]) * mult if size[-1] in "KMG" else int(size)
    return {"cores_usable": cores, "cpu_model": model, "llc_bytes": llc, "llc_instances": len(seen)}


def cpu_baseline(w, info: dict, budget_s: float = 8.0) -> dict:
    """The oracle's graft (numpy scatter of payload pages through a block table) timed on the
    host, on a bounded sample of the workload's artifact: the first L_s layers of a 4,096-token
    block, L_s chosen so that the payload alone is at least 1 GiB and four times the last-level
    cache the usable cores reach (so the copy streams from DRAM).  Timed single-threaded, then with one thread per usable
    core grafting its own slice of the block's pages (numpy releases the interpreter lock
    inside its copy loops).  Beside it, the oracle's fp64 attention per unit, with BLAS limited to one
    thread and with BLAS on every core."""
    import threading

    import numpy as np

    from oracle.paging import PagedPool, graft as o_graft
    block = w.block_tokens or w.prefix
    n_pages = w.pages_for(block)
    per_layer = 2 * n_pages * w.n_kv_heads * w.page_size * w.head_dim * 2
    layers = min(w.n_layers, max(-(-(1 << 30) // per_layer), -(-4 * info["llc_bytes"] // per_layer)))
    rng = np.random.default_rng(0)
    payload = np.empty((layers, 2, n_pages, w.n_kv_heads, w.page_size, w.head_dim), dtype=np.uint16)
    payload.reshape(-1)[:] = np.arange(payload.size, dtype=np.uint64).astype(np.uint16)   # any bytes will do
    table = rng.permutation(n_pages + 8)[:n_pages]
    pool = PagedPool(layers, n_pages + 8, w.n_kv_heads, w.page_size, w.head_dim, "bf16")

    def timed(n_threads: int):
        # thread i grafts pages [p0, p1) of the block (every layer), through the same table
        bounds = np.linspace(0, n_pages, n_threads + 1).astype(int)
        parts = [(payload[:, :, a:b], table[a:b], (b - a) * w.page_size) for a, b in zip(bounds[:-1], bounds[1:])]
        reps, t = 0, 0.0
        t0 = time.perf_counter()
        while t < budget_s or reps == 0:
            ths = [threading.Thread(target=o_graft, args=(pool, pl, tb, 0, n)) for pl, tb, n in parts]
            for th in ths:
                th.start()
            for th in ths:
                th.join()
            reps += 1
            t = time.perf_counter() - t0
        return 2.0 * payload.nbytes * reps / t / 1e9, reps, t

    single, reps1, t1 = timed(1)
    n = info["cores_usable"]
    multi, repsn, tn = timed(n)
    sample = (f"oracle graft of the first {layers} of {w.n_layers} layers of a {block:,}-token block "
              f"({payload.nbytes / 2**20:.0f} MiB payload read and as much written per pass, last-level cache "
              f"{info['llc_bytes'] / 2**20:.0f} MiB): {repsn} passes in {tn:.1f} s on {n} threads "
              f"(one slice of the block's pages each); single thread {single:.1f} GB/s ({reps1} passes in {t1:.1f} s)")
    return {"value": round(multi, 3), "unit": "GB/s", "cores": n, "kind": "oracle", "sample": sample,
            "single_thread_GBps": round(single, 3), "host": info, "per_unit": oracle_attention_units(w)}


def oracle_attention_units(w, rows_sampled: int = 8):
    """The oracle's attention (fp64 numpy) timed per unit on layer 0 of the workload: one
    decode row (the last decode step's, over the whole context) and every 64th suffix row,
    on Gaussian inputs of the workload's shapes and scale (sigma 0.5, drawn with numpy's
    generator: the timing does not depend on the values), best of three calls, with BLAS on
    one thread and on all; extrapolated to the step's prefill row-layers and decode
    token-layers."""
    import numpy as np

    from oracle.attention import attend

    try:
        from threadpoolctl import threadpool_limits
    except ImportError:                                 # pragma: no cover
        threadpool_limits = None
    rng = np.random.default_rng(0)
    n_keys = w.ctx_final
    k = rng.standard_normal((n_keys, w.n_kv_heads, w.head_dim)) * 0.5
    v = rng.standard_normal((n_keys, w.n_kv_heads, w.head_dim)) * 0.5
    dec_row = np.array([n_keys - 1])
    suf_rows = w.prefix + np.arange(0, w.suffix, w.suffix // rows_sampled)
    qs = {name: rng.standard_normal((len(rows), w.n_q_heads, w.head_dim)) * 0.5
          for name, rows in (("decode", dec_row), ("prefill", suf_rows))}

    def run():
        out = {}
        for name, rows in (("decode", dec_row), ("prefill", suf_rows)):
            best = float("inf")
            for _ in range(3):                      # the first call also pays one-time set-up
                t0 = time.perf_counter()
                attend(qs[name], rows, k, v, w.scale, w.layer_window(0))
                best = min(best, time.perf_counter() - t0)
            out[name] = best / len(rows)
        return out

    res = {}
    if threadpool_limits is not None:
        with threadpool_limits(limits=1, user_api="blas"):
            res["blas_1_thread"] = run()
    res["blas_all_threads"] = run()
    fmt = {}
    for key, out in res.items():
        fmt[key] = {"prefill_row_layer_ms": round(out["prefill"] * 1e3, 3),
                    "decode_token_layer_ms": round(out["decode"] * 1e3, 3),
                    "step_attention_s_extrapolated": round(
                        (w.batch * w.suffix * out["prefill"] + w.batch * w.decode_steps * out["decode"]) * w.n_layers,
                        1)}
    fmt["blas_threads_all"] = _blas_threads()
    fmt["sample"] = (f"layer 0: decode row {int(dec_row[0])} over {n_keys} keys, {len(suf_rows)} suffix rows "
                     f"(every {w.suffix // rows_sampled}th), all {w.n_q_heads} heads; extrapolated to {w.batch} "
                     f"sequence(s) x {w.n_layers} layers")
    return fmt


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max((p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"), default=1)
    except Exception:
        return None


# ------------------------------------------------------------------------------ timing helpers
class Launches:
    """Event pairs around the launches of one phase on one stream."""

    def __init__(self, torch, stream):
        self.torch, self.stream, self.pairs = torch, stream, []

    def __enter__(self):
        self.e0 = self.torch.cuda.Event(enable_timing=True)
        self.e0.record(self.stream)
        return self

    def __exit__(self, *exc):
        e1 = self.torch.cuda.Event(enable_timing=True)
        e1.record(self.stream)
        self.pairs.append((self.e0, e1))

    def ms(self):
        return [a.elapsed_time(b) for a, b in self.pairs]


def mean(xs):
    return sum(xs) / len(xs)


# ------------------------------------------------------------------------------ 32k window (headline)
def window_bench(args) -> dict:
    """The 12B-class 32k window at batch 16 (the headline step, see the module docstring)."""
    import gc

    import torch

    from paper_2607_14431_amd import harness as h
    from paper_2607_14431_amd import kvg
    from synth import ROLE_K, ROLE_Q, ROLE_V
    from synth.gpu import raw_chunk
    from synth.workloads import WINDOW12B

    w = WINDOW12B
    stream = torch.cuda.current_stream()
    B, J, BT = w.batch, w.blocks_per_seq, w.block_tokens
    N, S, T = w.prefix, w.suffix, w.decode_steps
    seqs = list(range(B))
    rp = h.rope_of(w)

    # ---- setup (untimed): the batch's caches, each sequence's 8 store blocks grafted once
    g = h.new_arm(w, seqs, w.ctx_final, seed=300, poison_id=1)
    hdrs = [kvg.kvg_artifact_header_init(g.cache, BT, j * BT, rp) for j in range(J)]
    art_sha = None
    for bi, s in enumerate(seqs):
        for j in range(J):
            hdr, payload = h.store_artifact(w, w.seq_block(s, j), j)
            if art_sha is None:
                art_sha = h.sha256_tensor(payload)              # block (0, 0), checked after the steps
            h.graft(g, bi, hdr, payload, j * BT, j * BT)
            del payload
    torch.cuda.synchronize()
    ring = [torch.empty(hdrs[0].payload_bytes, dtype=torch.uint8, device="cuda") for _ in range(PAYLOAD_RING)]
    pairs = [(bi, j) for bi in range(B) for j in range(J)]
    q_s, k_s, v_s = (raw_chunk(w, r, seqs, N, S) for r in (ROLE_Q, ROLE_K, ROLE_V))
    meta_s = g.meta(N)
    ws_s = torch.empty(kvg.kvg_prefill_workspace_bytes(g.cache, meta_s, w.n_layers, S), dtype=torch.uint8,
                       device="cuda")
    out_s = torch.empty((w.n_layers, B, S, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    dec_in = [tuple(raw_chunk(w, r, seqs, N + S + i, 1)[:, :, 0].contiguous() for r in (ROLE_Q, ROLE_K, ROLE_V))
              for i in range(T)]
    meta_d = [g.meta(N + S + i) for i in range(T)]
    ws_d = kvg.decode_workspace(g.cache, meta_d[-1], w.n_layers)
    out_d = torch.empty((T, w.n_layers, B, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()

    dep, gra, pre, dec = (Launches(torch, stream) for _ in range(4))

    def step(record: bool):
        for i, (bi, j) in enumerate(pairs):
            buf = ring[i % PAYLOAD_RING]
            if record:
                with dep:
                    kvg.kvg_deposit(g.cache, g.tables[bi], j * BT, BT, buf, stream)
                with gra:
                    kvg.kvg_graft(g.cache, hdrs[j], buf, g.tables[bi], j * BT, j * BT, 0, stream)
            else:
                kvg.kvg_deposit(g.cache, g.tables[bi], j * BT, BT, buf, stream)
                kvg.kvg_graft(g.cache, hdrs[j], buf, g.tables[bi], j * BT, j * BT, 0, stream)
        if record:
            with pre:
                kvg.kvg_prefill_attn(g.cache, meta_s, rp, 0, w.n_layers, S, q_s, k_s, v_s, w.scale, out_s, ws_s,
                                     stream)
        else:
            kvg.kvg_prefill_attn(g.cache, meta_s, rp, 0, w.n_layers, S, q_s, k_s, v_s, w.scale, out_s, ws_s, stream)
        for i in range(T):
            q, k, v = dec_in[i]
            if record:
                with dec:
                    kvg.kvg_decode_attn(g.cache, meta_d[i], rp, 0, w.n_layers, q, k, v, w.scale, out_d[i], ws_d,
                                        stream)
            else:
                kvg.kvg_decode_attn(g.cache, meta_d[i], rp, 0, w.n_layers, q, k, v, w.scale, out_d[i], ws_d, stream)

    print(f"[bench] {w.name}: warmup {args.warmup}, timed steps {args.steps}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(True)
        torch.cuda.synchronize()
        print(f"[bench] {w.name}: step {i + 1}/{args.steps} done", file=sys.stderr, flush=True)
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    t_dep, t_gra, t_pre, t_dec = (mean(x.ms()) for x in (dep, gra, pre, dec))   # per launch

    # ---- verification (untimed): restored bytes and graft == fresh on a batch-1 fresh probe
    verdict = None
    if not args.no_verify:
        _, restored = h.deposit(g, 0, 0, BT, 0)
        same_art = h.sha256_tensor(restored) == art_sha
        del restored
        ring.clear()
        gc.collect()
        torch.cuda.empty_cache()
        verdict = same_art
        for bi in (0, B - 1):
            f = h.new_arm(w, [bi], w.ctx_final, seed=310 + bi, poison_id=0)
            h.fresh_prefix(f, append_only=True, chunk=BT)
            rf = h.continue_arm(f)
            torch.cuda.synchronize()
            verdict = verdict and h.bytes_equal(rf.suffix[:, 0], out_s[:, bi]) and \
                h.bytes_equal(rf.decode[:, :, 0], out_d[:, :, bi])
            del f, rf
            gc.collect()
            torch.cuda.empty_cache()
        print(f"[bench] {w.name}: graft == fresh {verdict}", file=sys.stderr, flush=True)

    pay = float(hdrs[0].payload_bytes)
    graft_gbps = 2.0 * pay / (t_gra * 1e-3) / 1e9
    deposit_gbps = 2.0 * pay / (t_dep * 1e-3) / 1e9
    dec_bytes = B * mean([decode_launch_bytes(w, N + S + i) for i in range(T)])
    dec_gbps = dec_bytes / (t_dec * 1e-3) / 1e9
    pf_flop = B * prefill_flops(w, N, S)
    pf_tflops = pf_flop / (t_pre * 1e-3) / 1e12
    out = {
        "ms_per_step": round(ms_step, 3), "value": round(graft_gbps, 1),
        "config": {"workload": w.name, "n_layers": w.n_layers, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "window_tokens": N, "blocks_per_window": J, "block_tokens": BT,
                   "store_blocks": w.store_blocks, "suffix": S, "decode_steps": T, "batch": B,
                   "page_size": w.page_size},
        "graft_eq_fresh": verdict,
        "decode_tok_s": round(B / (t_dec * 1e-3), 1),
        "decode_hbm_frac": round(dec_gbps / HBM_PEAK_GBPS, 4),
        "decode_ms_per_step": round(t_dec, 4),
        "deposit_GBps": round(deposit_gbps, 1),
        "prefill_TFLOPs": round(pf_tflops, 2),
        "phases_ms": {"deposit": round(t_dep * len(pairs), 3), "graft": round(t_gra * len(pairs), 3),
                      "prefill": round(t_pre, 3), "decode": round(t_dec * T, 3)},
        "roofline": {"kernel": "kvg_decode_attn: decode_kernel<bf16, 256, 2> + decode_merge_kernel",
                     "bound": "hbm", "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(dec_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": measured_traffic("traffic_12b_window32k.md", "decode_bytes_per_launch"),
                     "bytes_per_launch": round(dec_bytes), "avg_launch_us": round(t_dec * 1e3, 2)},
        "rooflines_other": {
            "graft_kernel": {"bound": "hbm", "achieved": round(graft_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                             "frac": round(graft_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": 2.0 * pay,
                             "launches_per_step": len(pairs), "avg_launch_us": round(t_gra * 1e3, 2),
                             "traffic": measured_traffic("traffic_12b_window32k.md", "graft_bytes_per_launch")},
            "deposit_kernel": {"bound": "hbm", "achieved": round(deposit_gbps, 1), "peak": HBM_PEAK_GBPS,
                               "unit": "GB/s", "frac": round(deposit_gbps / HBM_PEAK_GBPS, 4),
                               "bytes_per_launch": 2.0 * pay, "launches_per_step": len(pairs),
                               "avg_launch_us": round(t_dep * 1e3, 2)},
            "prefill (append + prefill_mfma_kernel, 16 x 512 rows)": {
                "bound": "mfma", "achieved": round(pf_tflops, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(pf_tflops / MFMA_BF16_PEAK_TFLOPS, 4), "flop_per_launch": pf_flop,
                "ms": round(t_pre, 3)},
        },
    }
    return out


# ------------------------------------------------------------------------------ 12B single block
def block_bench(args, steps: int, warmup: int, extras_on: bool) -> dict:
    """The 12B-class single-block step at batch 1: deposit of the 4,096-token block (gather),
    graft of the artifact into a second cache at its own position (scatter), suffix prefill on
    the grafted cache, 64 decode steps; with the figures taken after the steps (content digests,
    sliding windows, one-layer launches, the logit verdict, fp8 cache, relocation)."""
    import torch

    from paper_2607_14431_amd import harness as h
    from paper_2607_14431_amd import kvg
    from synth import ROLE_K, ROLE_Q, ROLE_V
    from synth.gpu import raw_chunk
    from synth.workloads import BLOCK12B, SWA12B

    w = BLOCK12B
    stream = torch.cuda.current_stream()
    N, S, T = w.prefix, w.suffix, w.decode_steps

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
    dep, gra, pre, dec = (Launches(torch, stream) for _ in range(4))

    def step(record: bool):
        with dep:
            kvg.kvg_deposit(fresh.cache, bt_fresh, 0, N, payload, stream)
        with gra:
            kvg.kvg_graft(graft_arm.cache, hdr, payload, bt_graft, 0, 0, 0, stream)
        with pre:
            kvg.kvg_prefill_attn(graft_arm.cache, meta_s, rp, 0, w.n_layers, S, q_s, k_s, v_s, w.scale, out_s, ws,
                                 stream)
        for i in range(T):
            q, k, v = dec_in[i]
            with dec:
                kvg.kvg_decode_attn(graft_arm.cache, meta_d[i], rp, 0, w.n_layers, q, k, v, w.scale, out_d[i],
                                    ws_dec, stream)
        if not record:
            for x in (dep, gra, pre, dec):
                x.pairs.clear()

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step(True)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    t_dep, t_gra, t_pre, t_dec = (mean(x.ms()) for x in (dep, gra, pre, dec))

    verdict = None
    res_fresh = res_graft = None
    if not args.no_verify:
        res_graft = (out_s.clone(), out_d.clone())
        _, restored = h.deposit(graft_arm, 0, 0, N, 0)
        res_fresh = h.continue_arm(fresh)
        torch.cuda.synchronize()
        verdict = (h.sha256_tensor(payload) == h.sha256_tensor(restored) and
                   h.bytes_equal(res_fresh.suffix, res_graft[0]) and h.bytes_equal(res_fresh.decode, res_graft[1]))

    graft_bytes = 2.0 * hdr.payload_bytes                     # payload read + pool written
    graft_gbps = graft_bytes / (t_gra * 1e-3) / 1e9
    deposit_gbps = graft_bytes / (t_dep * 1e-3) / 1e9
    dec_bytes = mean([decode_launch_bytes(w, N + S + i) for i in range(T)])
    dec_gbps = dec_bytes / (t_dec * 1e-3) / 1e9
    pf_flop = prefill_flops(w, N, S)
    pf_tflops = pf_flop / (t_pre * 1e-3) / 1e12
    extras = {}
    if extras_on:
        extras.update(digest_figures(kvg, torch, stream, w, payload, int(hdr.payload_bytes)))
        launches = dict(rp=rp, meta_s=meta_s, q_s=q_s, k_s=k_s, v_s=v_s, ws=ws, out_s=out_s, meta_d=meta_d,
                        dec_in=dec_in, ws_dec=ws_dec, out_d=out_d)
        extras.update(window_figures(kvg, torch, stream, w, graft_arm.cache, launches, SWA12B.layer_windows))
        extras.update(per_layer_figures(kvg, torch, stream, w, graft_arm.cache, launches))
        extras.update(logit_figures(h, kvg, torch, stream, w, res_fresh, res_graft))
        extras.update(fp8_figures(h, kvg, torch, stream, w))
        extras.update(relocation_figures(h, kvg, torch, stream, w, hdr, payload))
    return {
        "config": {"workload": w.name, "n_layers": w.n_layers, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "block_tokens": N, "suffix": S, "decode_steps": T, "batch": w.batch},
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms_step, 3),
        "graft_eq_fresh": verdict,
        "graft_GBps": round(graft_gbps, 1), "graft_hbm_frac": round(graft_gbps / HBM_PEAK_GBPS, 4),
        "deposit_GBps": round(deposit_gbps, 1), "deposit_hbm_frac": round(deposit_gbps / HBM_PEAK_GBPS, 4),
        "decode_tok_s": round(w.batch / (t_dec * 1e-3), 1), "decode_hbm_frac": round(dec_gbps / HBM_PEAK_GBPS, 4),
        "decode": {"bound": "hbm", "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                   "frac": round(dec_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": round(dec_bytes),
                   "avg_launch_us": round(t_dec * 1e3, 2),
                   "traffic": measured_traffic("traffic_12b_block4096.md", "decode_bytes_per_launch")},
        "prefill": {"bound": "mfma", "achieved": round(pf_tflops, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(pf_tflops / MFMA_BF16_PEAK_TFLOPS, 4), "flop_per_launch": pf_flop,
                    "ms": round(t_pre, 4)},
        "phases_ms": {"deposit": round(t_dep, 4), "graft": round(t_gra, 4), "prefill": round(t_pre, 4),
                      "decode": round(t_dec * T, 4)},
        "cold_prefill_ms": round(cold_ms, 2),
        "rooflines_other": extras,
    }


# ------------------------------------------------------------------------------ 31B relocated
def reloc_bench(args) -> dict:
    """The 31B-class block (60 layers, 32 / 16 heads, head_dim 128, 16,384 tokens) captured at
    position 0 by 8 sequences and grafted 8,192 positions further (keys re-rotated by the
    offset), then the 8 sequences' 1,024-token suffix prefill and 64 decode steps, each launch
    timed with events.  Beside it (untimed): the own-position graft == fresh on one sequence,
    and the relocation residual against a fresh computation at +8,192 with the graft-free
    control (fresh at 0 against fresh at +8,192), Sec. 4.2."""
    import gc

    import torch

    from paper_2607_14431_amd import harness as h
    from paper_2607_14431_amd import kvg
    from synth import ROLE_K, ROLE_Q, ROLE_V
    from synth.gpu import raw_chunk
    from synth.workloads import RELOC31B, scaled

    stream = torch.cuda.current_stream()
    w0 = scaled(RELOC31B, start_pos=0)
    w = RELOC31B
    d = w.start_pos - w.own_pos
    seqs = list(range(w.batch))
    N, S, T, B = w.prefix, w.suffix, w.decode_steps, w.batch
    fresh = h.new_arm(w0, seqs, w0.ctx_final, seed=400, poison_id=0)
    h.fresh_prefix(fresh, append_only=True, chunk=4096)
    arts = [h.deposit(fresh, bi, 0, w0.prefix, 0) for bi in range(B)]
    del fresh
    gc.collect()
    torch.cuda.empty_cache()
    g = h.new_arm(w, seqs, w.ctx_final, seed=402, poison_id=1)
    gra = Launches(torch, stream)
    for rep in range(2):                                  # the first pass pays first-touch costs
        for bi, (hdr, payload) in enumerate(arts):
            with gra:
                h.graft(g, bi, hdr, payload, 0, w.start_pos, relocate=True)
        torch.cuda.synchronize()
        if rep == 0:
            gra.pairs.clear()
    t_gra = mean(gra.ms())
    pay = float(arts[0][0].payload_bytes)
    rp = h.rope_of(w)
    q_s, k_s, v_s = (raw_chunk(w, r, seqs, N, S) for r in (ROLE_Q, ROLE_K, ROLE_V))
    meta_s = g.meta(N)
    ws_s = torch.empty(kvg.kvg_prefill_workspace_bytes(g.cache, meta_s, w.n_layers, S), dtype=torch.uint8,
                       device="cuda")
    out_s = torch.empty((w.n_layers, B, S, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    pre = Launches(torch, stream)
    for rep in range(4):                                  # rewrites the same K/V bytes
        with pre:
            kvg.kvg_prefill_attn(g.cache, meta_s, rp, 0, w.n_layers, S, q_s, k_s, v_s, w.scale, out_s, ws_s, stream)
    torch.cuda.synchronize()
    t_pre = sorted(pre.ms()[1:])[1]                       # median of the last three
    del q_s, k_s, v_s, ws_s
    dec = Launches(torch, stream)
    ws_d = kvg.decode_workspace(g.cache, g.meta(N + S + T - 1), w.n_layers)
    out_d = torch.empty((T, w.n_layers, B, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    for i in range(T):
        q, k, v = (raw_chunk(w, r, seqs, N + S + i, 1)[:, :, 0].contiguous() for r in (ROLE_Q, ROLE_K, ROLE_V))
        with dec:
            kvg.kvg_decode_attn(g.cache, g.meta(N + S + i), rp, 0, w.n_layers, q, k, v, w.scale, out_d[i], ws_d,
                                stream)
    torch.cuda.synchronize()
    t_dec = mean(dec.ms())
    graft_gbps = 2.0 * pay / (t_gra * 1e-3) / 1e9
    dec_bytes = B * mean([decode_launch_bytes(w, N + S + i) for i in range(T)])
    dec_gbps = dec_bytes / (t_dec * 1e-3) / 1e9
    pf_flop = B * prefill_flops(w, N, S)
    out = {
        "config": {"workload": w.name, "n_layers": w.n_layers, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "block_tokens": N, "relocated_by": d, "suffix": S, "decode_steps": T,
                   "batch": B},
        "relocated_graft": {"bound": "hbm", "achieved": round(graft_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                            "frac": round(graft_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": 2.0 * pay,
                            "ms_per_launch": round(t_gra, 4), "launches": len(gra.pairs)},
        "prefill": {"bound": "mfma", "achieved": round(pf_flop / (t_pre * 1e-3) / 1e12, 1),
                    "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(pf_flop / (t_pre * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4), "flop": pf_flop,
                    "ms": round(t_pre, 3)},
        "decode": {"bound": "hbm", "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                   "frac": round(dec_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": round(dec_bytes),
                   "ms_per_step": round(t_dec, 3), "tok_s": round(B / (t_dec * 1e-3), 1)},
    }
    if not args.no_verify:
        # sequence 0 at batch 1: own-position graft == fresh, and the residual of the
        # relocated outputs against fresh at +d beside the graft-free control
        w1, wd1 = scaled(w0, batch=1), scaled(w, batch=1)
        f0 = h.new_arm(w1, [0], w1.ctx_final, seed=410, poison_id=0)
        h.fresh_prefix(f0, append_only=True, chunk=4096)
        r_f0 = h.continue_arm(f0)
        del f0
        g0 = h.new_arm(w1, [0], w1.ctx_final, seed=411, poison_id=1)
        h.graft(g0, 0, arts[0][0], arts[0][1], 0, 0)
        r_g0 = h.continue_arm(g0)
        del g0
        fd = h.new_arm(wd1, [0], wd1.ctx_final, seed=412, poison_id=0)
        h.fresh_prefix(fd, append_only=True, chunk=4096)
        _, k_fresh = h.deposit(fd, 0, 0, N, d)
        r_fd = h.continue_arm(fd)
        del fd
        _, k_moved = h.deposit(g, 0, 0, N, d)
        torch.cuda.synchronize()
        half = k_moved.numel() // (2 * w.n_layers)
        km = k_moved.view(w.n_layers, 2, half)[:, 0].reshape(-1).view(torch.int16)
        kf = k_fresh.view(w.n_layers, 2, half)[:, 0].reshape(-1).view(torch.int16)
        rel = torch.cat([out_s[:, 0].reshape(-1), out_d[:, :, 0].reshape(-1)])
        fr_d = torch.cat([r_fd.suffix[:, 0].reshape(-1), r_fd.decode[:, :, 0].reshape(-1)])
        fr_0 = torch.cat([r_f0.suffix[:, 0].reshape(-1), r_f0.decode[:, :, 0].reshape(-1)])
        out["own_position_graft_eq_fresh"] = h.bytes_equal(r_g0.suffix, r_f0.suffix) and \
            h.bytes_equal(r_g0.decode, r_f0.decode)
        out["relocation_residual"] = {
            "offset": d, "keys_differing_frac": round((km != kf).float().mean().item(), 4),
            "output_max_abs_vs_fresh_at_offset": float((rel - fr_d).abs().max().item()),
            "graft_free_control_max_abs": float((fr_0 - fr_d).abs().max().item()),
            "byte_exact": bool(torch.equal(rel.view(torch.int32), fr_d.view(torch.int32)))}
    return out


# ------------------------------------------------------------------------------ 2.85M-token store
STORE_DEPTH_BLOCKS = (0, 81, 169, 344, 520, 607, 688, 696)   # the paper's needle depths + the partial last block


def store_bench(args) -> dict:
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
    from synth import ROLE_K, ROLE_Q, ROLE_V
    from synth.gpu import raw_chunk
    from synth.workloads import STORE12B

    stream = torch.cuda.current_stream()
    w = STORE12B
    win = h.StoreWindow(w)
    pinned = h.PinnedPayload(h.kvg.kvg_payload_bytes(win.cache, w.block_tokens))
    for b in range(win.slots, 2 * win.slots):       # initial window fill (untimed)
        win.graft(b, win.materialize(b, pinned), pinned)
    torch.cuda.synchronize()
    kvg = h.kvg
    arm, N, S, T = win.arm, win.win_tokens, w.suffix, w.decode_steps
    rows = []
    for b in STORE_DEPTH_BLOCKS:
        hdr = win.materialize(b, pinned)
        vw = view_after(win, b)
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
        print(f"[bench] store access block {b}: {rows[-1]}", file=sys.stderr, flush=True)
    full = [r for r in rows if r["block_tokens"] == w.block_tokens]
    return {
        "config": {"workload": w.name, "store_tokens": w.store_tokens, "store_blocks": w.store_blocks,
                   "window_slots": win.slots, "batch": win.batch, "suffix": w.suffix, "decode_steps": w.decode_steps},
        "metric": "store access latency vs depth (graft from host + suffix prefill + decode)",
        "mean_access_ms": round(mean([r["access_ms"] for r in full]), 3), "higher_is_better": False,
        "max_over_min_graft_ms": round(max(r["graft_ms"] for r in full) / min(r["graft_ms"] for r in full), 3),
        "depths": rows,
    }


def view_after(win, b):
    """The window's workload view once block b has been grafted into its slot (the history
    entry is added by the graft itself; the view is needed before, to build the inputs)."""
    j = b % win.slots
    win.history[j].append((b, win.w.store_block_tokens(b)))
    vw = win.view()
    win.history[j].pop()
    return vw


# ------------------------------------------------------------------------------ tiny fp32
def tiny_bench() -> dict:
    """The tiny fp32 case (1 layer, 4 / 2 heads, head_dim 64, 256-token block): graft == fresh
    over five trials, each with its own page permutations and poison."""
    import torch

    from paper_2607_14431_amd import harness as h
    from synth.workloads import TINY

    w = TINY
    equal = 0
    for trial in range(5):
        f = h.new_arm(w, [0], w.ctx_final, seed=100 + trial, poison_id=0)
        h.fresh_prefix(f)
        hdr, payload = h.deposit(f, 0, 0, w.prefix, 0)
        rf = h.continue_arm(f)
        g = h.new_arm(w, [0], w.ctx_final, seed=200 + trial, poison_id=1)
        h.graft(g, 0, hdr, payload, 0, 0)
        rg = h.continue_arm(g)
        torch.cuda.synchronize()
        equal += int(rf.digest() == rg.digest())
    return {"config": {"workload": w.name}, "graft_eq_fresh": equal == 5, "trials_sha256_equal": equal,
            "trials": 5}


# ------------------------------------------------------------------------------ main
def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (this build has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return

    from synth.workloads import WINDOW12B
    cpu = None
    if args.workload in ("all", "12b-window32k") and not args.no_cpu_baseline:
        # on the host's cores, before the first GPU call
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(WINDOW12B, host_info())

    import torch
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    if args.workload in ("12b-block4096", "31b-reloc16k", "12b-store2.85M"):
        fn = {"12b-block4096": lambda: block_bench(args, args.steps, args.warmup, not args.no_extras),
              "31b-reloc16k": lambda: reloc_bench(args), "12b-store2.85M": lambda: store_bench(args)}
        print(json.dumps(fn[args.workload]()), flush=True)
        return

    head = window_bench(args)
    import gc
    gc.collect()
    torch.cuda.empty_cache()
    line = {
        "metric": "graft restore GB/s; decode-attn tok/s over grafted ctx (% HBM peak); graft==fresh",
        "value": head["value"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic", "config": head["config"],
    }
    line.update({k: v for k, v in head.items() if k not in ("value", "ms_per_step", "config")})
    copy_gbps = measured_copy_gbps(torch, stream)
    line["runtime_copy_GBps"] = round(copy_gbps, 1)             # hipMemcpy-class D2D copy of 1 GiB
    line["roofline"]["frac_of_runtime_copy"] = round(line["roofline"]["achieved"] / copy_gbps, 4)
    if args.workload == "all" and not args.no_extras:
        configs = {}
        for name, fn in (("12b-block4096", lambda: block_bench(args, 10, 3, True)),
                         ("31b-reloc16k", lambda: reloc_bench(args)),
                         ("12b-store2.85M", lambda: store_bench(args)),
                         ("tiny-f32", tiny_bench)):
            print(f"[bench] configuration {name}", file=sys.stderr, flush=True)
            configs[name] = fn()
            gc.collect()
            torch.cuda.empty_cache()
        line["configs"] = configs
    if cpu is not None:
        line["cpu_baseline"] = cpu
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
    step): one graft_relocate_kernel launch re-rotates the keys by the offset and copies the
    values, into a scratch cache.  Algorithmic bytes: the payload read and the pages
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
    return {"relocated graft, +8,192 positions (graft_relocate_kernel, not in the step)": {
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
