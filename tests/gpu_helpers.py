"""Host/device conversions for the GPU tests (test infrastructure)."""

import numpy as np
import torch


TORCH_DTYPE = {"bf16": torch.bfloat16, "f32": torch.float32, "fp8": torch.float8_e4m3fn}
NP_BITS = {"bf16": np.uint16, "f32": np.uint32, "fp8": np.uint8}
INT_VIEW = {"bf16": torch.int16, "f32": torch.int32, "fp8": torch.uint8}
RAW_DTYPE = {"bf16": "bf16", "f32": "f32", "fp8": "bf16"}    # raw inputs of a cache dtype


def bits_to_device(bits: np.ndarray, dtype: str) -> torch.Tensor:
    """numpy storage bits -> device tensor of the storage dtype (same bytes)."""
    if dtype == "bf16":
        return torch.from_numpy(bits.astype(np.uint16).view(np.int16)).cuda().view(torch.bfloat16)
    if dtype == "fp8":
        return torch.from_numpy(bits.astype(np.uint8)).cuda().view(torch.float8_e4m3fn)
    return torch.from_numpy(bits.astype(np.uint32).view(np.int32)).cuda().view(torch.float32)


def device_to_bits(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> numpy storage bits (uint16 for bf16, uint32 for fp32, uint8 otherwise)."""
    t = t.contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.view(torch.int32).cpu().numpy().view(np.uint32)
    if t.dtype == torch.float8_e4m3fn:
        return t.view(torch.uint8).cpu().numpy()
    return t.cpu().numpy()


def pair_norm(x: np.ndarray, pairing: int = 0) -> np.ndarray:
    """Norm of each element's rotary pair (0: i with i + D/2; 1: 2i with 2i + 1), per element."""
    D = x.shape[-1]
    if pairing == 0:
        r = np.sqrt(x[..., : D // 2] ** 2 + x[..., D // 2:] ** 2)
        return np.concatenate([r, r], axis=-1)
    r = np.sqrt(x[..., 0::2] ** 2 + x[..., 1::2] ** 2)
    return np.repeat(r, 2, axis=-1)


def ulp(x: np.ndarray, dtype: str) -> np.ndarray:
    """Spacing of the storage grid at x (fp8 E4M3: 4 significant bits, fixed 2^-9 below 2^-6)."""
    bits = {"bf16": 8, "f32": 24, "fp8": 4}[dtype]
    u = np.ldexp(1.0, np.frexp(np.maximum(np.abs(x), 1e-30))[1] - bits)
    return np.maximum(u, 2.0 ** -9) if dtype == "fp8" else u


def assert_rotated_close(got: np.ndarray, want: np.ndarray, raw_norm: np.ndarray, dtype: str):
    """GPU keys (fp32 rotation, one rounding) vs oracle keys (fp64 rotation, one rounding):
    at most one storage ulp apart, plus the fp32 rotation error (a few 2^-24 of the pair
    norm) where cancellation makes the value itself tiny."""
    tol = ulp(want, dtype) * 1.0001 + 4.0 * 2.0 ** -24 * raw_norm
    bad = np.abs(got - want) > tol
    assert not bad.any(), (f"{bad.sum()} elements beyond 1 ulp; first at {np.argwhere(bad)[0]}: "
                           f"got {got[bad][0]} want {want[bad][0]}")


def attention_close(got: np.ndarray, want: np.ndarray, dtype: str):
    """Tolerance of the attention outputs against the fp64 oracle: max-abs 1e-5 (fp32 caches) or
    2e-2 (bf16 caches), plus relative Frobenius 1e-6 / 1e-2 so that small outputs are not
    passed vacuously."""
    max_abs = float(np.max(np.abs(got - want)))
    rel = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-300))
    lim_abs, lim_rel = (1e-5, 1e-6) if dtype == "f32" else (2e-2, 1e-2)
    assert np.all(np.isfinite(got)), "non-finite output"
    assert max_abs <= lim_abs, f"max-abs {max_abs:.3e} > {lim_abs}"
    assert rel <= lim_rel, f"rel-Frobenius {rel:.3e} > {lim_rel}"
    return max_abs, rel
