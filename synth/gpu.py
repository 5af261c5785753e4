"""ctypes wrapper of the GPU input generator (libkvg_synth.so, built from gen.hip).

Produces the same bits as ``synth.philox.normal_tensor`` for the same (seed, stream,
index); tests check that on sampled elements.
"""

from __future__ import annotations

import ctypes
import os

import torch

from .philox import TOKEN_STRIDE  # noqa: F401  (the index layout gen.hip implements)
from .workloads import Workload

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvg_synth.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_14431_amd.build`")
_lib = ctypes.CDLL(LIB_PATH)
_lib.synth_fill.restype = ctypes.c_int
_lib.synth_fill.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
                            ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_uint64, ctypes.c_uint64,
                            ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]


def fill(dst: torch.Tensor, layer_stride: int, n_layers: int, layer_id0: int, t0: int, n_tokens: int,
         n_heads: int, head_dim: int, seed: int, stream_id: int, sigma_log2: int, bf16: bool, stream=None):
    """dst: a device tensor whose data_ptr is element (layer 0, token 0, head 0, dim 0)."""
    s = torch.cuda.current_stream() if stream is None else stream
    rc = _lib.synth_fill(ctypes.c_void_p(dst.data_ptr()), layer_stride, n_layers, layer_id0, t0, n_tokens, n_heads,
                         head_dim, seed, stream_id, sigma_log2, int(bf16), ctypes.c_void_p(s.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"synth_fill failed: {rc}")


def raw_chunk(w: Workload, role: int, seqs, t0: int, n_tokens: int, layers=None, sigma_log2=None,
              out: torch.Tensor | None = None) -> torch.Tensor:
    """Raw inputs [n_layers][len(seqs)][n_tokens][H][D] for logical tokens [t0, t0 + n_tokens)
    of the given sequences, in the workload's storage dtype, on the current device."""
    from .philox import ROLE_Q
    layers = list(range(w.n_layers)) if layers is None else list(layers)
    H = w.n_q_heads if role == ROLE_Q else w.n_kv_heads
    D = w.head_dim
    dt = torch.bfloat16 if w.raw_dtype == "bf16" else torch.float32
    B = len(seqs)
    if out is None:
        out = torch.empty((len(layers), B, n_tokens, H, D), dtype=dt, device="cuda")
    sig = w.sigma_log2 if sigma_log2 is None else sigma_log2
    layer_stride = B * n_tokens * H * D
    assert layers == list(range(layers[0], layers[0] + len(layers))), "layers must be contiguous"
    from .philox import ROLE_K, ROLE_NK, ROLE_NV, ROLE_V
    from .workloads import NEEDLE_SIGMA_LOG2
    for bi, s in enumerate(seqs):
        for (a, cnt, unit, off) in w.segments(s):
            lo, hi = max(a, t0), min(a + cnt, t0 + n_tokens)
            if lo >= hi:
                continue
            dst = out[0, bi, lo - t0]
            fill(dst, layer_stride, len(layers), layers[0], off + (lo - a), hi - lo, H, D, w.seed,
                 w.stream(role, unit).id, sig, w.raw_dtype == "bf16")
            tn = w.needle_at(unit, off + (lo - a), hi - lo) if role in (ROLE_K, ROLE_V) else None
            if tn is not None:
                # the store block's needle row replaces the token's row (same bits as the numpy side)
                nrole = ROLE_NK if role == ROLE_K else ROLE_NV
                fill(out[0, bi, lo - t0 + tn - (off + (lo - a))], layer_stride, len(layers), layers[0], 0, 1, H, D,
                     w.seed, w.stream(nrole, unit).id, NEEDLE_SIGMA_LOG2, w.raw_dtype == "bf16")
    return out
