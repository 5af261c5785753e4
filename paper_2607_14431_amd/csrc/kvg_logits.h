// Logit head and logit comparison: device argument blocks and host-side launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvg {

constexpr int kLogitKBlock = 128;     // hidden elements per pipelined step pair (two 64-element blocks)

constexpr int kPackRows = 128;        // rows per packed block

// Fragment-major packing of a [n][H] bf16 matrix, n zero-padded to a multiple of 128: the
// 16-byte unit (B, kb, m, t, lane) -- B = row / 128, m = (row / 32) % 4, kb = k / 64,
// t in 0..3, lane in 0..63 -- holds row 128 B + 32 m + lane % 32, elements
// 64 kb + 32 (lane / 32) + 8 t .. + 8.  Unit index ((((B * H / 64) + kb) * 4 + m) * 4 + t)
// * 64 + lane: one MFMA operand fragment of a wave (fixed B, kb, m, t) is 1 KiB of
// consecutive bytes, the fragments of a 128-row block for one 64-element step are 16 KiB in a
// row, and the block's whole hidden range is one contiguous run.  `b32` is the 32-row block
// index 4 B + m.
__host__ __device__ inline int64_t packed_unit(int64_t b32, int64_t kb, int t, int lane, int64_t n_kb) {
  return ((((b32 >> 2) * n_kb + kb) * 4 + (b32 & 3)) * 4 + t) * 64 + lane;
}

__host__ __device__ inline int64_t packed_rows(int64_t n) { return (n + kPackRows - 1) / kPackRows * kPackRows; }

struct LogitArgs {
  const float* hidden;       // [rows][H] fp32
  uint16_t* hidden_packed;   // workspace: bf16 hidden, packed, rows_pad rows (padding zero)
  const uint16_t* w_packed;  // packed bf16 weights, packed_rows(V) rows
  float* out;                // [rows][V] fp32
  int32_t rows, rows_pad, H, V;
  float cap;                 // soft cap; 0 = none
};

struct PackArgs {
  const uint16_t* w;         // [V][H] bf16, row-major
  uint16_t* packed;          // packed_rows(V) rows, packed (rows past V zero)
  int32_t V, H;
};

struct CompareArgs {
  const float* a;            // [rows][V] fp32
  const float* b;            // [rows][V] fp32
  int32_t rows, V;
  double* kl;                // [rows]
  int32_t* arg_a;            // [rows]
  int32_t* arg_b;            // [rows]
};

hipError_t launch_logits(const LogitArgs& a, hipStream_t stream);
hipError_t launch_logits_pack(const PackArgs& a, hipStream_t stream);
hipError_t launch_logit_compare(const CompareArgs& a, hipStream_t stream);

}  // namespace kvg
