"""Chunked-prefill and decode attention (bf16 MFMA path and fp32 VALU path) against the oracle with
ragged chunks, per-sequence context lengths that are not tile multiples, several query
tiles, GQA groups 1/2/4 and a peaky variant (queries scaled x8 plus diagonal needles) whose
outputs are far above the tolerance.  Sliding-window layers (row i sees keys (i - W, i],
Sec. 4.3's windowed layers) run beside global ones, with windows of one key, windows that end
inside a key tile (64) or a decode split (512), and windows longer than the context.  Both
rotary pairings (half split and interleaved) on every path."""

import numpy as np
import pytest
import torch

from oracle.attention import attend
from oracle.numerics import bits_to_values, round_to
from oracle.rope import rotate
from synth import ROLE_K, ROLE_Q, ROLE_V, normal_tensor
from synth.philox import Stream

from gpu_helpers import INT_VIEW, RAW_DTYPE, TORCH_DTYPE, attention_close, bits_to_device

pytestmark = pytest.mark.gpu

CASES = [
    # dtype, D, Hq, Hkv, ctx_lens per sequence, chunk, q sigma_log2, needle divisor
    ("bf16", 256, 4, 2, [0, 77, 600], 130, -1, 0),
    ("bf16", 128, 4, 4, [64, 1000], 200, -1, 0),
    ("bf16", 128, 8, 2, [5, 300], 33, -1, 0),
    ("bf16", 64, 2, 1, [129], 257, -1, 0),
    ("bf16", 256, 4, 2, [300, 17], 96, 2, 8),     # peaky: q sigma 4, needles k = q / 8
    ("bf16", 256, 4, 2, [300, 17], 96, 2, 2),     # harsh: needles k = q / 2, score std ~8
    ("bf16", 128, 8, 2, [700, 3], 70, 2, 2),      # harsh, group 4, D 128 (8 waves)
    ("bf16", 128, 16, 2, [600, 40], 90, 2, 2),    # harsh, group 8 (vector ALU path)
    ("f32", 64, 4, 2, [33, 250], 40, 0, 0),
    ("f32", 64, 4, 2, [100], 24, 3, 8),           # peaky fp32
    # fp8 E4M3 caches (bf16 inputs): MFMA for groups 1, 2, 4 at D 256, 128, 64; VALU for group 8
    ("fp8", 256, 4, 2, [0, 77, 600], 130, -1, 0),
    ("fp8", 128, 4, 4, [64, 1000], 200, -1, 0),
    ("fp8", 64, 2, 1, [129], 257, -1, 0),
    ("fp8", 128, 16, 4, [300, 5], 150, -1, 0),
    ("fp8", 128, 16, 2, [600, 40], 90, -1, 0),
    ("fp8", 256, 4, 2, [300, 17], 96, 2, 8),      # peaky fp8
    ("fp8", 256, 4, 2, [300, 17], 96, 2, 2),      # harsh fp8
]


def _gen(role, s, t0, n, L, H, D, sig, dtype):
    return normal_tensor(77, Stream(30, role, s), range(L), t0, n, H, D, sig, dtype)


def _needle_bits(q_bits, div, dtype):
    """Raw key bits equal to a raw query row divided by a power of two (exact in bf16 and fp32)."""
    qv = bits_to_values(q_bits, dtype) / div
    return (np.asarray(qv, np.float32).view(np.uint32) >> (16 if dtype == "bf16" else 0)).astype(q_bits.dtype)


@pytest.mark.parametrize("dtype,D,Hq,Hkv,ctxs,chunk,qsig,div", CASES)
def test_prefill_matches_oracle(dtype, D, Hq, Hkv, ctxs, chunk, qsig, div):
    _prefill_case(dtype, D, Hq, Hkv, ctxs, chunk, qsig, (0, 0), div)


WINDOW_CASES = [
    # dtype, D, Hq, Hkv, ctx_lens, chunk, windows per layer (3 layers)
    ("bf16", 256, 4, 2, [0, 700], 130, (100, 0, 1)),          # MFMA group 2
    ("bf16", 128, 4, 4, [77, 1000], 200, (64, 513, 5000)),     # MFMA group 1
    ("bf16", 128, 16, 4, [300], 150, (250, 0, 37)),            # MFMA group 4
    ("bf16", 128, 16, 2, [600, 40], 90, (600, 65, 0)),         # VALU group 8
    ("f32", 64, 4, 2, [1100, 3], 45, (512, 1, 700)),           # fp32 VALU
    ("fp8", 256, 4, 2, [0, 700], 130, (100, 0, 1)),           # fp8 MFMA
]


@pytest.mark.parametrize("dtype,D,Hq,Hkv,ctxs,chunk,windows", WINDOW_CASES)
def test_prefill_window_matches_oracle(dtype, D, Hq, Hkv, ctxs, chunk, windows):
    _prefill_case(dtype, D, Hq, Hkv, ctxs, chunk, -1 if dtype == "bf16" else 0, windows)


def _prefill_case(dtype, D, Hq, Hkv, ctxs, chunk, qsig, windows, div=0, pairing="half"):
    from paper_2607_14431_amd import kvg
    L, B = len(windows), len(ctxs)
    store, dtype = dtype, RAW_DTYPE[dtype]          # cache dtype; dtype of the raw inputs
    kv_sig = -1 if dtype == "bf16" else 0
    max_ctx = max(ctxs)
    per_seq = (max_ctx + chunk + 15) // 16
    n_pages = B * per_seq + 5
    rng = np.random.default_rng(D * 7 + chunk)
    tables = rng.permutation(n_pages)[: B * per_seq].reshape(B, per_seq).astype(np.int32)
    cache = kvg.Cache.allocate(L, n_pages, Hq, Hkv, D, TORCH_DTYPE[store], windows=windows)
    cache.k_pool.view(INT_VIEW[store]).fill_(0x7F if store == "fp8" else 0x7FC1)
    cache.v_pool.view(INT_VIEW[store]).fill_(0x7F if store == "fp8" else 0x7FC1)
    start = np.array([1000 * (i + 1) for i in range(B)], dtype=np.int64)
    tb = torch.from_numpy(tables).cuda()
    rp = kvg.rope(10000.0, {"half": kvg.KVG_ROPE_HALF, "interleaved": kvg.KVG_ROPE_INTERLEAVED}[pairing])
    # prefixes: one append per sequence (different lengths)
    for b, c in enumerate(ctxs):
        if c == 0:
            continue
        kb = _gen(ROLE_K, b, 0, c, L, Hkv, D, kv_sig, dtype)
        vb = _gen(ROLE_V, b, 0, c, L, Hkv, D, kv_sig, dtype)
        seqs1 = kvg.Seqs(tb[b:b + 1], torch.zeros(1, dtype=torch.int32, device="cuda"),
                         torch.from_numpy(start[b:b + 1]).cuda(), 0)
        kvg.kvg_append(cache, seqs1, rp, 0, L, c, bits_to_device(kb[:, None], dtype),
                       bits_to_device(vb[:, None], dtype))
    # the chunk for all sequences at once
    q = np.stack([_gen(ROLE_Q, b, c, chunk, L, Hq, D, qsig, dtype) for b, c in enumerate(ctxs)], axis=1)
    k = np.stack([_gen(ROLE_K, b, c, chunk, L, Hkv, D, kv_sig, dtype) for b, c in enumerate(ctxs)], axis=1)
    v = np.stack([_gen(ROLE_V, b, c, chunk, L, Hkv, D, kv_sig, dtype) for b, c in enumerate(ctxs)], axis=1)
    if div:
        # diagonal needles: the key of every 5th row is its first query head / div.  With
        # div 8 the needle keys have the sigma of the others (off-diagonal scores std ~2);
        # with div 2 they are four times larger, so a row's scores against the other rows'
        # needle keys have a standard deviation of ~8 (a peaked softmax whose weights move
        # with the last bits of the scores) and the diagonal score is ~|q|^2 / (2 sqrt(D))
        for b in range(B):
            for i in range(0, chunk, 5):
                for g in range(Hkv):
                    k[:, b, i, g] = _needle_bits(q[:, b, i, g * (Hq // Hkv)], div, dtype)
    seqs = kvg.Seqs(tb, torch.tensor(ctxs, dtype=torch.int32, device="cuda"), torch.from_numpy(start).cuda(), max_ctx)
    out = torch.empty((L, B, chunk, Hq, D), dtype=torch.float32, device="cuda")
    ws = torch.empty(kvg.kvg_prefill_workspace_bytes(cache, seqs, L, chunk), dtype=torch.uint8, device="cuda")
    kvg.kvg_prefill_attn(cache, seqs, rp, 0, L, chunk, bits_to_device(q, dtype), bits_to_device(k, dtype),
                         bits_to_device(v, dtype), 1.0 / np.sqrt(D), out, ws)
    torch.cuda.synchronize()
    got_all = out.cpu().numpy().astype(np.float64)
    for b, c in enumerate(ctxs):
        n = c + chunk
        kr = np.concatenate([_gen(ROLE_K, b, 0, c, L, Hkv, D, kv_sig, dtype), k[:, b]], axis=1) if c else k[:, b]
        vr = np.concatenate([_gen(ROLE_V, b, 0, c, L, Hkv, D, kv_sig, dtype), v[:, b]], axis=1) if c else v[:, b]
        pos = start[b] + np.arange(n)
        K = round_to(rotate(bits_to_values(kr, dtype), pos, 10000.0, pairing), store)
        V = round_to(bits_to_values(vr, dtype), store)
        Q = rotate(bits_to_values(q[:, b], dtype), pos[c:], 10000.0, pairing)
        for li in range(L):
            want = attend(Q[li], np.arange(c, n), K[li], V[li], 1.0 / np.sqrt(D), windows[li])
            max_abs, rel = attention_close(got_all[li, b], want, store)
            print(f"seq {b} layer {li} window {windows[li]}: max-abs {max_abs:.2e} rel {rel:.2e} "
                  f"max|ref| {np.abs(want).max():.3f}")
            if div:
                assert np.abs(want).max() > 0.2, "peaky case is not peaky"


DECODE_CASES = [
    # dtype, D, Hq, Hkv, ctx_lens, steps, q sigma_log2, needle divisor
    ("bf16", 256, 4, 2, [510, 1023, 5], 4, -1, 0),
    ("bf16", 128, 8, 4, [1536, 64], 3, -1, 0),
    ("f32", 64, 4, 2, [511, 2], 3, 0, 0),
    ("bf16", 256, 4, 2, [1300, 40], 4, 2, 2),     # harsh: q sigma 4, needles k = q / 2
    ("bf16", 128, 16, 2, [900, 17], 3, 2, 2),     # harsh, group 8
    ("bf16", 256, 4, 2, [1300, 40], 4, 3, 2),     # harsher: q sigma 8 (bf16-rounded queries: ~7e-2)
    ("bf16", 256, 4, 2, [0, 1, 513], 3, -1, 0),   # empty and one-token caches, a split boundary
    ("f32", 64, 4, 2, [0, 511], 2, 0, 0),
    # fp8 E4M3 caches (bf16 inputs, keys and values rounded once when stored)
    ("fp8", 256, 4, 2, [510, 1023, 5], 4, -1, 0),
    ("fp8", 128, 16, 2, [1536, 64], 3, -1, 0),    # group 8
    ("fp8", 256, 4, 2, [1300, 40], 4, 2, 2),      # harsh fp8
]


@pytest.mark.parametrize("dtype,D,Hq,Hkv,ctxs,steps,qsig,div", DECODE_CASES)
def test_decode_matches_oracle(dtype, D, Hq, Hkv, ctxs, steps, qsig, div):
    """Decode over several consecutive steps on one workspace: per-sequence contexts that
    cross the 512-key split boundaries, oracle parity.  The harsh cases plant needle keys:
    every 5th cached key is the query its row would have had, halved (q sigma 4, so a decode
    query's scores against those keys have a standard deviation of ~8), and every other
    decode step's own key is its query halved (the step retrieves its own value)."""
    _decode_case(dtype, D, Hq, Hkv, ctxs, steps, (0, 0), qsig, div)


DECODE_WINDOW_CASES = [
    # windows that start in the middle of a page, exactly on a split boundary, that leave
    # one split, several splits, or only the new token; and one longer than every context
    ("bf16", 256, 4, 2, [510, 1023, 1600], 3, (1, 512, 700)),
    ("bf16", 128, 8, 4, [1536, 64, 2100], 3, (1000, 17, 4096)),
    ("f32", 64, 4, 2, [1030, 2], 3, (513, 0, 2)),
]


@pytest.mark.parametrize("dtype,D,Hq,Hkv,ctxs,steps,windows", DECODE_WINDOW_CASES)
def test_decode_window_matches_oracle(dtype, D, Hq, Hkv, ctxs, steps, windows):
    _decode_case(dtype, D, Hq, Hkv, ctxs, steps, windows)


def _decode_case(dtype, D, Hq, Hkv, ctxs, steps, windows, qsig=None, div=0, pairing="half"):
    from paper_2607_14431_amd import kvg
    L, B = len(windows), len(ctxs)
    store, dtype = dtype, RAW_DTYPE[dtype]          # cache dtype; dtype of the raw inputs
    kv_sig = -1 if dtype == "bf16" else 0
    qsig = kv_sig if qsig is None else qsig
    G = Hq // Hkv

    def keys(b, n):
        """Raw keys [L][n][Hkv][D] of sequence b, needles planted."""
        kr = _gen(ROLE_K, b, 0, n, L, Hkv, D, kv_sig, dtype)
        if div:
            qr = _gen(ROLE_Q, b, 0, n, L, Hq, D, qsig, dtype)
            c = ctxs[b]
            needle_rows = list(range(0, c, 5)) + [c + i for i in range(0, steps, 2) if c + i < n]
            for j in needle_rows:
                for g in range(Hkv):
                    kr[:, j, g] = _needle_bits(qr[:, j, g * G], div, dtype)
        return kr
    max_ctx = max(ctxs) + steps
    per_seq = (max_ctx + 15) // 16
    n_pages = B * per_seq + 3
    rng = np.random.default_rng(D + steps)
    tables = rng.permutation(n_pages)[: B * per_seq].reshape(B, per_seq).astype(np.int32)
    cache = kvg.Cache.allocate(L, n_pages, Hq, Hkv, D, TORCH_DTYPE[store], windows=windows)
    cache.k_pool.view(INT_VIEW[store]).fill_(0x7F if store == "fp8" else 0x7FC1)
    cache.v_pool.view(INT_VIEW[store]).fill_(0x7F if store == "fp8" else 0x7FC1)
    start = np.array([7 * (i + 1) for i in range(B)], dtype=np.int64)
    tb = torch.from_numpy(tables).cuda()
    st_dev = torch.from_numpy(start).cuda()
    rp = kvg.rope(10000.0, {"half": kvg.KVG_ROPE_HALF, "interleaved": kvg.KVG_ROPE_INTERLEAVED}[pairing])
    all_k = [keys(b, c + steps) for b, c in enumerate(ctxs)]
    for b, c in enumerate(ctxs):
        if c == 0:                  # an empty cache: the first step attends to its own token only
            continue
        kb = all_k[b][:, :c]
        vb = _gen(ROLE_V, b, 0, c, L, Hkv, D, kv_sig, dtype)
        seqs1 = kvg.Seqs(tb[b:b + 1], torch.zeros(1, dtype=torch.int32, device="cuda"), st_dev[b:b + 1], 0)
        kvg.kvg_append(cache, seqs1, rp, 0, L, c, bits_to_device(np.ascontiguousarray(kb[:, None]), dtype),
                       bits_to_device(vb[:, None], dtype))
    seqs0 = kvg.Seqs(tb, torch.tensor(ctxs, dtype=torch.int32, device="cuda"), st_dev, max_ctx)
    ws = kvg.decode_workspace(cache, seqs0, L)
    outs = []
    for i in range(steps):
        lens = [c + i for c in ctxs]
        q = np.stack([_gen(ROLE_Q, b, c, 1, L, Hq, D, qsig, dtype)[:, 0] for b, c in enumerate(lens)], axis=1)
        k = np.stack([all_k[b][:, c] for b, c in enumerate(lens)], axis=1)
        v = np.stack([_gen(ROLE_V, b, c, 1, L, Hkv, D, kv_sig, dtype)[:, 0] for b, c in enumerate(lens)], axis=1)
        seqs = kvg.Seqs(tb, torch.tensor(lens, dtype=torch.int32, device="cuda"), st_dev, max(lens))
        out = torch.empty((L, B, Hq, D), dtype=torch.float32, device="cuda")
        kvg.kvg_decode_attn(cache, seqs, rp, 0, L, bits_to_device(q, dtype), bits_to_device(k, dtype),
                            bits_to_device(v, dtype), 1.0 / np.sqrt(D), out, ws)
        outs.append(out)
    torch.cuda.synchronize()
    for b, c in enumerate(ctxs):
        n = c + steps
        kr = all_k[b]
        vr = _gen(ROLE_V, b, 0, n, L, Hkv, D, kv_sig, dtype)
        qr = _gen(ROLE_Q, b, c, steps, L, Hq, D, qsig, dtype)
        pos = start[b] + np.arange(n)
        K = round_to(rotate(bits_to_values(kr, dtype), pos, 10000.0, pairing), store)
        V = round_to(bits_to_values(vr, dtype), store)
        Q = rotate(bits_to_values(qr, dtype), pos[c:], 10000.0, pairing)
        got = np.stack([o[:, b].cpu().numpy() for o in outs], axis=1).astype(np.float64)   # [L][steps][Hq][D]
        for li in range(L):
            want = attend(Q[li], np.arange(c, n), K[li], V[li], 1.0 / np.sqrt(D), windows[li])
            max_abs, rel = attention_close(got[li], want, store)
            print(f"decode seq {b} layer {li} window {windows[li]}: max-abs {max_abs:.2e} rel {rel:.2e} "
                  f"max|ref| {np.abs(want).max():.3f}")
            if div:
                assert np.abs(want).max() > 0.2, "peaky case is not peaky"


def test_decode_bytes_do_not_depend_on_the_batch():
    """A sequence's decode output is the same bytes alone (3 splits in the workspace) and
    beside a sequence long enough that the workspace holds more than 16 splits, which the
    merge combines with its general loop instead of one round of loads; on a global and a
    windowed layer."""
    from paper_2607_14431_amd import kvg
    dtype, D, Hq, Hkv, windows = "bf16", 128, 4, 2, (0, 700)
    L, ctxs = len(windows), [1500, 9000]
    per_seq = (max(ctxs) + 1 + 15) // 16
    tables = np.random.default_rng(5).permutation(2 * per_seq).reshape(2, per_seq).astype(np.int32)
    cache = kvg.Cache.allocate(L, 2 * per_seq, Hq, Hkv, D, torch.bfloat16, windows=windows)
    cache.k_pool.view(torch.int16).fill_(0x7FC1)
    cache.v_pool.view(torch.int16).fill_(0x7FC1)
    tb = torch.from_numpy(tables).cuda()
    st = torch.tensor([3, 11], dtype=torch.int64, device="cuda")
    rp = kvg.rope(10000.0)
    for b, c in enumerate(ctxs):
        kb = _gen(ROLE_K, b, 0, c, L, Hkv, D, -1, dtype)
        vb = _gen(ROLE_V, b, 0, c, L, Hkv, D, -1, dtype)
        seqs1 = kvg.Seqs(tb[b:b + 1], torch.zeros(1, dtype=torch.int32, device="cuda"), st[b:b + 1], 0)
        kvg.kvg_append(cache, seqs1, rp, 0, L, c, bits_to_device(kb[:, None], dtype), bits_to_device(vb[:, None], dtype))
    raw = [np.stack([_gen(role, b, c, 1, L, H, D, -1, dtype)[:, 0] for b, c in enumerate(ctxs)], axis=1)
           for role, H in ((ROLE_Q, Hq), (ROLE_K, Hkv), (ROLE_V, Hkv))]
    both = kvg.Seqs(tb, torch.tensor(ctxs, dtype=torch.int32, device="cuda"), st, max(ctxs))
    ws = kvg.decode_workspace(cache, both, L)
    outs = []
    for B in (2, 1):
        seqs = kvg.Seqs(tb[:B], torch.tensor(ctxs[:B], dtype=torch.int32, device="cuda"), st[:B], max(ctxs[:B]))
        q, k, v = (bits_to_device(np.ascontiguousarray(x[:, :B]), dtype) for x in raw)
        out = torch.empty((L, B, Hq, D), dtype=torch.float32, device="cuda")
        kvg.kvg_decode_attn(cache, seqs, rp, 0, L, q, k, v, 1.0 / np.sqrt(D), out, ws)
        outs.append(out)
    torch.cuda.synchronize()
    assert torch.equal(outs[0][:, 0].view(torch.int32), outs[1][:, 0].view(torch.int32))


SHARED_CASES = [
    # cache dtype, head_dim, query heads, KV heads
    ("bf16", 128, 4, 2),       # 8 waves per workgroup, group 2
    ("bf16", 256, 8, 2),       # 4 waves per workgroup, group 4
    ("fp8", 128, 4, 4),        # fp8 pages widened to bf16, group 1
]


@pytest.mark.parametrize("store,D,Hq,Hkv", SHARED_CASES)
def test_decode_shared_window_splits(store, D, Hq, Hkv):
    """40 sequences decoding over one shared 1,920-token window (identical leading block-table
    entries) plus private tails.  With kvg_seqs.shared_tokens set, the window's whole 512-key
    splits of the full-attention layer come from the shared-split kernel (every sequence's
    query against each shared page, read once, on MFMA) and the rest from the decode kernel;
    the windowed layer is all decode kernel.  Checked: the oracle on several sequences, the
    plain path within the same tolerance, the same bytes on a second call, and the plain
    path's own promise (a sequence alone gives the batch's bytes)."""
    from paper_2607_14431_amd import kvg
    dtype, windows = RAW_DTYPE[store], (0, 700)
    L, B, N = len(windows), 40, 1920
    tails = [1 + (7 * b) % 53 for b in range(B)]            # private tokens already cached
    shared_pages, priv_pages = N // 16, (max(tails) + 1 + 15) // 16
    n_pages = shared_pages + B * priv_pages
    perm = np.random.default_rng(9).permutation(n_pages).astype(np.int32)
    tables = np.empty((B, shared_pages + priv_pages), np.int32)
    tables[:, :shared_pages] = perm[:shared_pages]
    for b in range(B):
        tables[b, shared_pages:] = perm[shared_pages + b * priv_pages: shared_pages + (b + 1) * priv_pages]
    cache = kvg.Cache.allocate(L, n_pages, Hq, Hkv, D, TORCH_DTYPE[store], windows=windows)
    cache.k_pool.view(INT_VIEW[store]).fill_(0x7F if store == "fp8" else 0x7FC1)
    cache.v_pool.view(INT_VIEW[store]).fill_(0x7F if store == "fp8" else 0x7FC1)
    tb = torch.from_numpy(tables).cuda()
    st = torch.zeros(B, dtype=torch.int64, device="cuda")
    rp = kvg.rope(10000.0)
    kw = _gen(ROLE_K, 0, 0, N, L, Hkv, D, -1, dtype)           # the shared window, written once
    vw = _gen(ROLE_V, 0, 0, N, L, Hkv, D, -1, dtype)
    seq0 = kvg.Seqs(tb[0:1], torch.zeros(1, dtype=torch.int32, device="cuda"), st[0:1], 0)
    kvg.kvg_append(cache, seq0, rp, 0, L, N, bits_to_device(kw[:, None], dtype), bits_to_device(vw[:, None], dtype))
    kt_bits, vt_bits = [], []
    for b, t in enumerate(tails):                            # each sequence's private tail
        kt = _gen(ROLE_K, b + 1, N, t, L, Hkv, D, -1, dtype)
        vt = _gen(ROLE_V, b + 1, N, t, L, Hkv, D, -1, dtype)
        kt_bits.append(kt)
        vt_bits.append(vt)
        sb = kvg.Seqs(tb[b:b + 1], torch.full((1,), N, dtype=torch.int32, device="cuda"), st[b:b + 1], N)
        kvg.kvg_append(cache, sb, rp, 0, L, t, bits_to_device(kt[:, None], dtype), bits_to_device(vt[:, None], dtype))
    ctxs = [N + t for t in tails]
    raw = [np.stack([_gen(role, b + 1, c, 1, L, H, D, -1, dtype)[:, 0] for b, c in enumerate(ctxs)], axis=1)
           for role, H in ((ROLE_Q, Hq), (ROLE_K, Hkv), (ROLE_V, Hkv))]
    q, k, v = (bits_to_device(np.ascontiguousarray(x), dtype) for x in raw)
    lens = torch.tensor(ctxs, dtype=torch.int32, device="cuda")
    outs = []
    for hint in (0, N, N):
        seqs = kvg.Seqs(tb, lens, st, max(ctxs), hint)
        ws = kvg.decode_workspace(cache, seqs, L)
        out = torch.full((L, B, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
        kvg.kvg_decode_attn(cache, seqs, rp, 0, L, q, k, v, 1.0 / np.sqrt(D), out, ws)
        outs.append(out)
    b1 = 5
    alone = kvg.Seqs(tb[b1:b1 + 1], lens[b1:b1 + 1], st[b1:b1 + 1], ctxs[b1])
    out1 = torch.empty((L, 1, Hq, D), dtype=torch.float32, device="cuda")
    q1, k1, v1 = (bits_to_device(np.ascontiguousarray(x[:, b1:b1 + 1]), dtype) for x in raw)
    kvg.kvg_decode_attn(cache, alone, rp, 0, L, q1, k1, v1, 1.0 / np.sqrt(D), out1, kvg.decode_workspace(cache, alone, L))
    torch.cuda.synchronize()
    plain, shared, again = (o.cpu().numpy().astype(np.float64) for o in outs)
    assert np.all(np.isfinite(shared))
    assert torch.equal(outs[1].view(torch.int32), outs[2].view(torch.int32)), "shared path not deterministic"
    assert torch.equal(outs[0][:, b1].view(torch.int32), out1[:, 0].view(torch.int32))
    # layer 0 is full attention: its shared splits take the MFMA path (bf16 P), so its bytes
    # differ from the plain path's
    assert not torch.equal(outs[0][0].view(torch.int32), outs[1][0].view(torch.int32)), "shared path not taken"
    print("shared vs plain:", attention_close(shared, plain, store))
    for b in (0, b1, B - 1):
        c = ctxs[b]
        kb = np.concatenate([kw, kt_bits[b], raw[1][:, b][:, None]], axis=1)
        vb = np.concatenate([vw, vt_bits[b], raw[2][:, b][:, None]], axis=1)
        pos = np.arange(c + 1, dtype=np.float64)
        K = round_to(rotate(bits_to_values(kb, dtype), pos, 10000.0), store)
        V = round_to(bits_to_values(vb, dtype), store)
        Q = rotate(bits_to_values(raw[0][:, b][:, None], dtype), pos[c:], 10000.0)
        for li in range(L):
            want = attend(Q[li], np.array([c]), K[li], V[li], 1.0 / np.sqrt(D), windows[li])[0]
            print(f"seq {b} layer {li}:", attention_close(shared[li, b], want, store))


@pytest.mark.parametrize("store,D,Hq,Hkv", SHARED_CASES)
def test_prefill_shared_window_splits(store, D, Hq, Hkv):
    """A 29-row suffix prefill for each of 12 sequences over one shared 1,600-token window
    plus private tails.  With kvg_seqs.shared_tokens set, the full-attention layer's keys in
    the window's whole 512-key splits ([0, 1536)) come from the shared-split kernel (the
    batch's rows against each shared page, read once) and the rest ([1536, ctx + row]) from
    the per-sequence kernel, the two partials combined; the windowed layer is all
    per-sequence kernel.  Checked: the oracle on several sequences, the plain path within
    the tolerance (the same bytes on the windowed layer), the same bytes on a second call."""
    from paper_2607_14431_amd import kvg
    dtype, windows = RAW_DTYPE[store], (0, 700)
    L, B, N, C = len(windows), 12, 1600, 29                 # C below every case's row tile
    tails = [1 + (11 * b) % 47 for b in range(B)]            # private tokens already cached
    shared_pages, priv_pages = N // 16, (max(tails) + C + 15) // 16
    n_pages = shared_pages + B * priv_pages
    perm = np.random.default_rng(10).permutation(n_pages).astype(np.int32)
    tables = np.empty((B, shared_pages + priv_pages), np.int32)
    tables[:, :shared_pages] = perm[:shared_pages]
    for b in range(B):
        tables[b, shared_pages:] = perm[shared_pages + b * priv_pages: shared_pages + (b + 1) * priv_pages]
    cache = kvg.Cache.allocate(L, n_pages, Hq, Hkv, D, TORCH_DTYPE[store], windows=windows)
    cache.k_pool.view(INT_VIEW[store]).fill_(0x7F if store == "fp8" else 0x7FC1)
    cache.v_pool.view(INT_VIEW[store]).fill_(0x7F if store == "fp8" else 0x7FC1)
    tb = torch.from_numpy(tables).cuda()
    st = torch.zeros(B, dtype=torch.int64, device="cuda")
    rp = kvg.rope(10000.0)
    kw = _gen(ROLE_K, 0, 0, N, L, Hkv, D, -1, dtype)           # the shared window, written once
    vw = _gen(ROLE_V, 0, 0, N, L, Hkv, D, -1, dtype)
    seq0 = kvg.Seqs(tb[0:1], torch.zeros(1, dtype=torch.int32, device="cuda"), st[0:1], 0)
    kvg.kvg_append(cache, seq0, rp, 0, L, N, bits_to_device(kw[:, None], dtype), bits_to_device(vw[:, None], dtype))
    kt_bits, vt_bits = [], []
    for b, t in enumerate(tails):
        kt = _gen(ROLE_K, b + 1, N, t, L, Hkv, D, -1, dtype)
        vt = _gen(ROLE_V, b + 1, N, t, L, Hkv, D, -1, dtype)
        kt_bits.append(kt)
        vt_bits.append(vt)
        sb = kvg.Seqs(tb[b:b + 1], torch.full((1,), N, dtype=torch.int32, device="cuda"), st[b:b + 1], N)
        kvg.kvg_append(cache, sb, rp, 0, L, t, bits_to_device(kt[:, None], dtype), bits_to_device(vt[:, None], dtype))
    ctxs = [N + t for t in tails]
    raw = [np.stack([_gen(role, b + 1, c, C, L, H, D, -1, dtype) for b, c in enumerate(ctxs)], axis=1)
           for role, H in ((ROLE_Q, Hq), (ROLE_K, Hkv), (ROLE_V, Hkv))]
    q, k, v = (bits_to_device(np.ascontiguousarray(x), dtype) for x in raw)
    lens = torch.tensor(ctxs, dtype=torch.int32, device="cuda")
    outs = []
    for hint in (0, N, N):
        seqs = kvg.Seqs(tb, lens, st, max(ctxs), hint)
        ws = torch.empty(kvg.kvg_prefill_workspace_bytes(cache, seqs, L, C), dtype=torch.uint8, device="cuda")
        out = torch.full((L, B, C, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
        kvg.kvg_prefill_attn(cache, seqs, rp, 0, L, C, q, k, v, 1.0 / np.sqrt(D), out, ws)
        outs.append(out)
    torch.cuda.synchronize()
    plain, shared, again = (o.cpu().numpy().astype(np.float64) for o in outs)
    assert np.all(np.isfinite(shared))
    assert torch.equal(outs[1].view(torch.int32), outs[2].view(torch.int32)), "shared path not deterministic"
    assert torch.equal(outs[0][1].view(torch.int32), outs[1][1].view(torch.int32)), "windowed layer changed"
    assert not torch.equal(outs[0][0].view(torch.int32), outs[1][0].view(torch.int32)), "shared path not taken"
    print("shared vs plain:", attention_close(shared, plain, store))
    for b in (0, 5, B - 1):
        c = ctxs[b]
        kb = np.concatenate([kw, kt_bits[b], raw[1][:, b]], axis=1)
        vb = np.concatenate([vw, vt_bits[b], raw[2][:, b]], axis=1)
        pos = np.arange(c + C, dtype=np.float64)
        K = round_to(rotate(bits_to_values(kb, dtype), pos, 10000.0), store)
        V = round_to(bits_to_values(vb, dtype), store)
        Q = rotate(bits_to_values(raw[0][:, b], dtype), pos[c:], 10000.0)
        for li in range(L):
            want = attend(Q[li], np.arange(c, c + C), K[li], V[li], 1.0 / np.sqrt(D), windows[li])
            print(f"seq {b} layer {li}:", attention_close(shared[li, b], want, store))


INTERLEAVED_CASES = [
    # the rotary pairing (2i, 2i + 1): MFMA (bf16, fp8), vector (fp32, group 8) prefill
    ("bf16", 256, 4, 2, [77, 600], 130),
    ("bf16", 128, 16, 2, [5, 300], 33),
    ("fp8", 128, 4, 4, [64, 1000], 200),
    ("f32", 64, 4, 2, [33, 250], 40),
]


@pytest.mark.parametrize("dtype,D,Hq,Hkv,ctxs,chunk", INTERLEAVED_CASES)
def test_prefill_interleaved_matches_oracle(dtype, D, Hq, Hkv, ctxs, chunk):
    _prefill_case(dtype, D, Hq, Hkv, ctxs, chunk, -1 if dtype != "f32" else 0, (0, 0), pairing="interleaved")


@pytest.mark.parametrize("dtype,D,Hq,Hkv,ctxs,steps", [("bf16", 256, 4, 2, [510, 1023, 5], 3),
                                                       ("fp8", 128, 16, 2, [1536, 64], 2),
                                                       ("f32", 64, 4, 2, [511, 2], 3)])
def test_decode_interleaved_matches_oracle(dtype, D, Hq, Hkv, ctxs, steps):
    _decode_case(dtype, D, Hq, Hkv, ctxs, steps, (0, 0), pairing="interleaved")
