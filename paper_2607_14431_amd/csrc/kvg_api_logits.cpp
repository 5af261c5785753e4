// C ABI of the logit head and the logit comparison (declarations and contracts in
// include/kvg.h).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kvg.h"
#include "kvg_logits.h"

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

int32_t rows_pad(int32_t rows) { return (int32_t)kvg::packed_rows(rows); }

bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

}  // namespace

extern "C" {

size_t kvg_logits_packed_bytes(int32_t vocab, int32_t hidden) {
  if (vocab <= 0 || hidden <= 0) return 0;
  return (size_t)kvg::packed_rows(vocab) * hidden * sizeof(uint16_t);
}

int kvg_logits_pack(const uint16_t* w_dev, int32_t vocab, int32_t hidden, uint16_t* packed_dev, void* stream) {
  if (w_dev == nullptr || packed_dev == nullptr || vocab <= 0 || hidden <= 0) return KVG_E_INVAL;
  if (hidden % kvg::kLogitKBlock != 0) return KVG_E_SHAPE;
  if (!aligned16(w_dev) || !aligned16(packed_dev)) return KVG_E_ALIGN;
  kvg::PackArgs a;
  a.w = w_dev;
  a.packed = packed_dev;
  a.V = vocab;
  a.H = hidden;
  return kvg::launch_logits_pack(a, static_cast<hipStream_t>(stream)) == hipSuccess ? KVG_OK : KVG_E_HIP;
}

size_t kvg_logits_workspace_bytes(int32_t rows, int32_t hidden) {
  if (rows <= 0 || hidden <= 0) return 0;
  return align_up((size_t)rows_pad(rows) * hidden * sizeof(uint16_t));
}

int kvg_logits(const float* hidden_dev, int32_t rows, int32_t hidden, const uint16_t* w_packed_dev, int32_t vocab,
               float cap, float* logits_dev, void* ws_dev, size_t ws_bytes, void* stream) {
  if (hidden_dev == nullptr || w_packed_dev == nullptr || logits_dev == nullptr || rows <= 0 || hidden <= 0 ||
      vocab <= 0 || !(cap >= 0.0f) || !std::isfinite(cap))
    return KVG_E_INVAL;
  if (hidden % kvg::kLogitKBlock != 0) return KVG_E_SHAPE;
  if ((int64_t)rows * vocab > INT64_MAX / 4 || (int64_t)vocab * hidden > INT64_MAX / 2) return KVG_E_SHAPE;
  if (!aligned16(hidden_dev) || !aligned16(w_packed_dev) || !aligned16(logits_dev)) return KVG_E_ALIGN;
  if (ws_dev == nullptr || ws_bytes < kvg_logits_workspace_bytes(rows, hidden)) return KVG_E_WORKSPACE;
  if (!aligned16(ws_dev)) return KVG_E_ALIGN;
  if (((int64_t)vocab + 127) / 128 * ((rows + 31) / 32) >= INT32_MAX) return KVG_E_SHAPE;
  kvg::LogitArgs a;
  a.hidden = hidden_dev;
  a.hidden_packed = static_cast<uint16_t*>(ws_dev);
  a.w_packed = w_packed_dev;
  a.out = logits_dev;
  a.rows = rows;
  a.rows_pad = rows_pad(rows);
  a.H = hidden;
  a.V = vocab;
  a.cap = cap;
  return kvg::launch_logits(a, static_cast<hipStream_t>(stream)) == hipSuccess ? KVG_OK : KVG_E_HIP;
}

int kvg_logit_compare(const float* a_dev, const float* b_dev, int32_t rows, int32_t vocab, double* kl_dev,
                      int32_t* argmax_a_dev, int32_t* argmax_b_dev, void* stream) {
  if (a_dev == nullptr || b_dev == nullptr || kl_dev == nullptr || argmax_a_dev == nullptr ||
      argmax_b_dev == nullptr || rows <= 0 || vocab <= 0)
    return KVG_E_INVAL;
  kvg::CompareArgs c;
  c.a = a_dev;
  c.b = b_dev;
  c.rows = rows;
  c.V = vocab;
  c.kl = kl_dev;
  c.arg_a = argmax_a_dev;
  c.arg_b = argmax_b_dev;
  return kvg::launch_logit_compare(c, static_cast<hipStream_t>(stream)) == hipSuccess ? KVG_OK : KVG_E_HIP;
}

}  // extern "C"
