// Logit head and logit comparison: device argument blocks and host-side launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvg {

constexpr int kLogitRowTile = 32;     // hidden rows per MFMA column block
constexpr int kLogitKBlock = 128;     // hidden elements per pipelined step pair (two 64-element blocks)

struct LogitArgs {
  const float* hidden;       // [rows][H] fp32
  uint16_t* hidden_bf16;     // workspace [rows_pad][H] bf16 (rows past `rows` zero)
  const uint16_t* w;         // [V][H] bf16
  float* out;                // [rows][V] fp32
  int32_t rows, rows_pad, H, V;
  float cap;                 // soft cap; 0 = none
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
hipError_t launch_logit_compare(const CompareArgs& a, hipStream_t stream);

}  // namespace kvg
