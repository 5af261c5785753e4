"""Storage rounding for the oracle (test infrastructure only).

The KV cache stores K and V in the workload's dtype.  The oracle computes in
fp64 and rounds once, to nearest with ties to even, when a value is stored.

fp8 storage (KV-cache quantization, which the paper lists among the serving settings
that shape a block, Sec. 4.4) is OCP FP8 E4M3: 1 sign, 4 exponent (bias 7), 3 mantissa
bits; normals down to 2^-6, subnormals in steps of 2^-9, largest finite 448, codes
0x7F / 0xFF NaN, no infinities.  Stored values saturate: |x| > 448 stores +-448.
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


FP8_MAX = 448.0
FP8_MIN_NORMAL = 2.0 ** -6
FP8_SUBNORMAL_STEP = 2.0 ** -9


def round_fp8(x: np.ndarray) -> np.ndarray:
    """fp64 -> nearest E4M3 value (ties to even), saturating at +-448, as fp64.

    Normals keep 4 significant bits (m * 2**e, m in [0.5, 1), rounded to m's 4 leading
    bits); below 2^-6 the grid is the fixed subnormal step 2^-9.  Signs (and -0) are kept.
    """
    x = np.clip(np.asarray(x, dtype=np.float64), -FP8_MAX, FP8_MAX)
    m, e = np.frexp(x)
    normal = np.ldexp(np.rint(np.ldexp(m, 4)), e - 4)
    sub = np.rint(x / FP8_SUBNORMAL_STEP) * FP8_SUBNORMAL_STEP
    out = np.where(np.abs(x) >= FP8_MIN_NORMAL, normal, sub)
    return np.copysign(out, x)


def fp8_bits_to_values(bits: np.ndarray) -> np.ndarray:
    """E4M3 codes (uint8) -> fp64 values; NaN codes give NaN."""
    b = np.asarray(bits).astype(np.int64)
    sign = np.where(b & 0x80, -1.0, 1.0)
    exp = (b >> 3) & 0xF
    man = b & 0x7
    val = np.where(exp == 0, man * FP8_SUBNORMAL_STEP, np.ldexp(1.0 + man / 8.0, exp - 7))
    val = np.where((b & 0x7F) == 0x7F, np.nan, val)
    return sign * val


def fp8_values_to_bits(x: np.ndarray) -> np.ndarray:
    """E4M3 values already on the grid (|x| <= 448) -> codes (uint8)."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(np.isnan(x)) or np.any(np.abs(x) > FP8_MAX) or np.any(round_fp8(x) != x):
        raise ValueError("value not representable in fp8 e4m3")
    sign = np.signbit(x).astype(np.int64) << 7
    a = np.abs(x)
    m, e = np.frexp(np.where(a >= FP8_MIN_NORMAL, a, 1.0))
    exp_field = np.where(a >= FP8_MIN_NORMAL, e - 1 + 7, 0)             # a = (2m) 2^(e-1)
    man_field = np.where(a >= FP8_MIN_NORMAL, np.rint((2 * m - 1) * 8), np.rint(a / FP8_SUBNORMAL_STEP))
    return (sign | (exp_field << 3) | man_field.astype(np.int64)).astype(np.uint8)


def round_f32(x: np.ndarray) -> np.ndarray:
    """fp64 -> nearest fp32 value (numpy's cast rounds to nearest even), as fp64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return round_f32(x)
    if dtype == "fp8":
        return round_fp8(x)
    raise ValueError(dtype)


def bits_to_values(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Storage bits (uint16 bf16 / uint32 fp32) -> fp64 values."""
    bits = np.asarray(bits)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f32":
        return bits.astype(np.uint32).view(np.float32).astype(np.float64)
    if dtype == "fp8":
        return fp8_bits_to_values(bits)
    raise ValueError(dtype)


def values_to_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp64 values already on the dtype's grid -> storage bits."""
    if dtype == "fp8":
        return fp8_values_to_bits(x)
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
    return {"bf16": np.uint16, "f32": np.uint32, "fp8": np.uint8}[dtype]
