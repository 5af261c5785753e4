"""Storage rounding for the oracle (test infrastructure only).

The KV cache stores K and V in the workload's dtype.  The oracle computes in
fp64 and rounds once, to nearest with ties to even, when a value is stored.
"""

from __future__ import annotations

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """fp64 -> nearest bf16 value (8 significant bits, ties to even), as fp64.

    x = m * 2**e with m in [0.5, 1); the bf16 value keeps m rounded to 8 bits.
    Zero stays zero.  Subnormal and overflow ranges are not reached by the
    workloads (|x| is far from 2**-126 and 2**127).
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def round_f32(x: np.ndarray) -> np.ndarray:
    """fp64 -> nearest fp32 value (numpy's cast rounds to nearest even), as fp64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return round_f32(x)
    raise ValueError(dtype)


def bits_to_values(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Storage bits (uint16 bf16 / uint32 fp32) -> fp64 values."""
    bits = np.asarray(bits)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f32":
        return bits.astype(np.uint32).view(np.float32).astype(np.float64)
    raise ValueError(dtype)


def values_to_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp64 values already on the dtype's grid -> storage bits."""
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    if not np.array_equal(x32.astype(np.float64), np.asarray(x, dtype=np.float64)):
        raise ValueError("value not representable in fp32")
    if dtype == "bf16":
        b = x32.view(np.uint32)
        if np.any(b & np.uint32(0xFFFF)):
            raise ValueError("value not representable in bf16")
        return (b >> np.uint32(16)).astype(np.uint16)
    if dtype == "f32":
        return x32.view(np.uint32)
    raise ValueError(dtype)


def storage_np_dtype(dtype: str):
    return {"bf16": np.uint16, "f32": np.uint32}[dtype]


def storage_bytes(dtype: str) -> int:
    return {"bf16": 2, "f32": 4}[dtype]
