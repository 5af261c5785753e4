// Device-side helpers and kernel parameter blocks shared by the libkvg kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvg {

constexpr int kPage = 16;           // tokens per page (the only supported page size)
constexpr int kMaxWindowLayers = 128;  // per-layer sliding windows a launch carries
constexpr int kSplit = 512;         // decode split-K range: 32 pages of logical index
constexpr int kMaxHalfDim = 128;    // head_dim <= 256

// ---- storage element traits -------------------------------------------------------
// bf16 is carried as its 16-bit pattern; conversion to fp32 is exact, conversion from
// fp32 rounds to nearest even (inputs are finite).
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b16) { return __uint_as_float(b16 << 16); }

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

template <typename T> struct Elem;

template <> struct Elem<uint16_t> {            // bf16 storage
  static constexpr int kPerVec = 8;            // elements per 16-byte vector
  __device__ static __forceinline__ float get(const uint4& v, int e) {
    const uint32_t w = (&v.x)[e >> 1];
    return (e & 1) ? __uint_as_float(w & 0xFFFF0000u) : __uint_as_float(w << 16);
  }
  __device__ static __forceinline__ void put(uint4& v, int e, float f) {
    uint32_t& w = (&v.x)[e >> 1];
    const uint32_t b = f32_to_bf16_bits(f);
    w = (e & 1) ? ((w & 0x0000FFFFu) | (b << 16)) : ((w & 0xFFFF0000u) | b);
  }
};

template <> struct Elem<float> {               // fp32 storage
  static constexpr int kPerVec = 4;
  __device__ static __forceinline__ float get(const uint4& v, int e) { return __uint_as_float((&v.x)[e]); }
  __device__ static __forceinline__ void put(uint4& v, int e, float f) { (&v.x)[e] = __float_as_uint(f); }
};

// Rotation of one pair with fp32 cos/sin.  The operation order is fixed:
//   a' = fma(a, c, -(b * s)),  b' = fma(a, s, b * c)
__device__ __forceinline__ void rotate_pair(float& a, float& b, float c, float s) {
  const float bs = b * s;
  const float bc = b * c;
  const float na = fmaf(a, c, -bs);
  const float nb = fmaf(a, s, bc);
  a = na;
  b = nb;
}

// ---- parameter blocks ----------------------------------------------------------------
struct AppendArgs {
  void* k_pool;
  void* v_pool;
  int64_t layer_elems;        // elements per layer in a pool = n_pages * Hkv * P * D
  int64_t n_pages;
  const int32_t* block_tables;
  const int32_t* ctx_lens;
  const int64_t* start_pos;
  const void* k_raw;          // [n_layers][batch][chunk][Hkv][D]
  const void* v_raw;
  const void* q_raw;          // [n_layers][batch][chunk][Hq][D] or null
  void* q_out;                // rotated queries, same layout, fp32 or bf16
  int32_t q_out_bf16;
  int32_t Hq, Hkv, D;
  int32_t layer0, n_layers, batch, chunk, max_pages, max_ctx_len;
  int32_t layers_per_block;
  int32_t pairing;            // 0 half, 1 interleaved
  double theta[kMaxHalfDim];  // base^(-2i/D) computed on the host in fp64
};

struct CopyArgs {
  void* k_pool;
  void* v_pool;
  int64_t layer_bytes;        // bytes per layer in a pool
  int64_t page_bytes;         // bytes of one page of one layer (Hkv * P * D * elem)
  int64_t n_pages;
  const int32_t* block_table; // the sequence's row
  void* payload;              // [L][2][n_block_pages][Hkv][P][D]
  int32_t first_page;
  int32_t n_block_pages;
  int32_t n_tokens;           // valid tokens in the block
  int32_t n_layers;
  int32_t row_bytes;          // D * elem
  int32_t Hkv, D;
  int32_t relocate;           // graft only: rotate keys by the table below
  int32_t pairing;
  float cs[2 * kMaxHalfDim];  // (cos, sin) of d * theta_i, fp64 on the host, rounded to fp32
};

struct AttnArgs {
  const void* k_pool;
  const void* v_pool;
  int64_t layer_elems;
  int64_t n_pages;
  const int32_t* block_tables;
  const int32_t* ctx_lens;
  const void* q;              // rotated queries [n_layers][batch][rows][Hq][D]: bf16 for bf16 caches, else fp32
  float* part_acc;            // [n_layers][batch][rows][Hq][n_split_max][D]
  float* part_ml;             // [n_layers][batch][rows][Hq][n_split_max][2]
  float* out;                 // [n_layers][batch][rows][Hq][D]
  float scale_log2;           // scale * log2(e)
  int32_t Hq, Hkv, D, group;
  int32_t layer0, n_layers, batch, rows, max_pages, max_ctx_len, n_split_max;
  int32_t window[kMaxWindowLayers];   // per layer of the launch: 0 = full causal, W = last W keys
};

struct DecodeArgs {
  void* k_pool;
  void* v_pool;
  int64_t layer_elems;
  int64_t n_pages;
  const int32_t* block_tables;
  const int32_t* ctx_lens;
  const int64_t* start_pos;
  const void* q_raw;          // [n_layers][batch][Hq][D] cache dtype, before rotation
  const void* k_raw;          // [n_layers][batch][Hkv][D]
  const void* v_raw;
  float* out;                 // [n_layers][batch][Hq][D]
  float* part_acc;            // [n_layers][batch][Hq][n_split_max][D]
  float* part_ml;             // [n_layers][batch][Hq][n_split_max][2]
  float scale_log2;
  int32_t Hq, Hkv, D, group;
  int32_t layer0, n_layers, batch, max_pages, max_ctx_len, n_split_max, pairing;
  double theta[kMaxHalfDim];
  int32_t window[kMaxWindowLayers];
};

struct PrefillArgs {
  const void* k_pool;
  const void* v_pool;
  int64_t layer_elems;
  int64_t n_pages;
  const int32_t* block_tables;
  const int32_t* ctx_lens;
  const uint16_t* q;          // rotated queries bf16 [n_layers][batch][chunk][Hq][D]
  float* out;                 // [n_layers][batch][chunk][Hq][D]
  float scale_log2;
  int32_t Hq, Hkv, D, group;
  int32_t layer0, n_layers, batch, chunk, max_pages, max_ctx_len, n_qt;
  int32_t window[kMaxWindowLayers];
};

// The window of layer l of a launch (0 beyond the carried range, which the host only
// allows when no layer is windowed).
template <typename Args>
__device__ __forceinline__ int layer_window(const Args& a, int l) {
  return l < kMaxWindowLayers ? a.window[l] : 0;
}

// First key a query sees when its causal prefix is keys [0, n_keys) and its layer's
// window is W (keys i - W < j <= i for the query at position i = n_keys - 1; W = 0 is
// full causal attention).
__device__ __forceinline__ int window_start(int W, int n_keys) {
  return W > 0 && n_keys > W ? n_keys - W : 0;
}

}  // namespace kvg
