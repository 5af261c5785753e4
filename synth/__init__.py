"""Seeded synthetic inputs shared by the HIP path and the CPU oracle.

This module generates raw (pre-RoPE) Q/K/V values and nothing else: it holds
none of the grafting or attention arithmetic.  Both sides draw their inputs
from here, the oracle through the numpy functions, the GPU path through the
HIP fill kernel in ``gen.hip`` (``libkvg_synth.so``); the two produce the same
bits for the same (seed, stream, index) and the tests check that they do.

Generator (stated once, implemented twice):

* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
  easy as 1, 2, 3", SC'11), counter = (index lo, index hi, stream lo,
  stream hi), key = (seed lo, seed hi).
* The four 32-bit output words give twelve 10-bit uniforms (bits 0-9, 10-19,
  20-29 of each word).  Their sum minus 6138 is an Irwin-Hall(12) integer
  z in [-6138, 6138] with mean 0 and variance 1024**2 - 1, so z / 1024 is a
  unit-variance, near-Gaussian value (range +-6 sigma, excess kurtosis -0.1).
* value = z * 2**(sigma_log2 - 10), exact in fp32 (|z| < 2**13).  sigma is a
  power of two, so N(0, 1) and N(0, 0.5) are exact choices.
* bf16 storage rounds that fp32 value to nearest-even (bit form below).

The integer construction is chosen so that the CPU and GPU sides agree bit for
bit without depending on any transcendental function.

Needles (the large store's planted facts, one per block): a workload with needles set
replaces, in every store block b, the key and value rows of one seeded token (for every
layer and KV head) by rows drawn from two streams of their own (roles NK and NV, unit =
the block's, sigma 1).  A probe query aimed at the needle key retrieves the needle value;
which key direction a probe needs is the test's business, not the generator's.
"""

from .philox import (  # noqa: F401
    PHILOX_M0, PHILOX_M1, PHILOX_W0, PHILOX_W1,
    philox4x32_10, irwin_hall12, normal_f32, f32_to_bf16_bits, bf16_bits_to_f32,
    normal_tensor, Stream, ROLE_Q, ROLE_K, ROLE_V, ROLE_W, ROLE_H, ROLE_NK, ROLE_NV, TOKEN_STRIDE,
)
