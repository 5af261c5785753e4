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

// storage dtype codes (the values of kvg_dtype)
constexpr int kDtypeF32 = 0, kDtypeBf16 = 1, kDtypeFp8 = 2;

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

// fp8 storage: OCP FP8 E4M3 (the chip's native fp8 conversions).  Stored values saturate at
// +-448 (the conversion instruction itself turns overflow into NaN); rounding is to nearest
// even, subnormals included.  The raw q/k/v handed to an fp8 cache are bf16.
constexpr float kFp8Max = 448.0f;

__device__ __forceinline__ float fp8_clamp(float f) { return fminf(fmaxf(f, -kFp8Max), kFp8Max); }

// two values into the low (HI = false) or high 16-bit half of `old`
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2(float a, float b, uint32_t old) {
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(fp8_clamp(a), fp8_clamp(b), (int)old, HI);
}

template <> struct Elem<uint8_t> {             // fp8 e4m3 storage
  static constexpr int kPerVec = 16;
  __device__ static __forceinline__ float get(const uint4& v, int e) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    const int w = (int)(&v.x)[e >> 2];
    const f32x2_t p = ((e >> 1) & 1) ? __builtin_amdgcn_cvt_pk_f32_fp8(w, true) : __builtin_amdgcn_cvt_pk_f32_fp8(w, false);
    return (e & 1) ? p.y : p.x;
  }
  __device__ static __forceinline__ void put(uint4& v, int e, float f) {
    uint32_t& w = (&v.x)[e >> 2];
    const uint32_t b = fp8x2<false>(f, 0.0f, 0u) & 0xFFu;
    const int sh = 8 * (e & 3);
    w = (w & ~(0xFFu << sh)) | (b << sh);
  }
};

// dtype of the raw inputs a cache of storage type T takes (fp8 caches take bf16)
template <typename T> struct RawOf { using type = T; };
template <> struct RawOf<uint8_t> { using type = uint16_t; };

// n consecutive values (a multiple of 4, at most 16) in storage type T, as 32-bit words
template <typename T, int N>
__device__ __forceinline__ void pack_words(const float* x, uint32_t* out) {
  if constexpr (sizeof(T) == 1) {
#pragma unroll
    for (int j = 0; j < N / 4; ++j)
      out[j] = fp8x2<true>(x[4 * j + 2], x[4 * j + 3], fp8x2<false>(x[4 * j], x[4 * j + 1], 0u));
  } else {
    uint4 v = make_uint4(0, 0, 0, 0);
    static_assert(N * sizeof(T) <= 16, "at most one vector");
#pragma unroll
    for (int e = 0; e < N; ++e) Elem<T>::put(v, e, x[e]);
#pragma unroll
    for (int j = 0; j < (int)(N * sizeof(T) / 4); ++j) out[j] = (&v.x)[j];
  }
}

// A rotated query value x as two bf16 values: hi = x rounded to nearest even, lo = the
// remainder x - hi (exact in fp32) rounded to nearest even.  hi + lo keeps 16 significant
// bits of x (relative error at most 2^-17), so a score accumulated from hi and lo products
// with bf16 keys is as accurate as an fp32-query score to within 2^-17 of the |q||k| sum.
__device__ __forceinline__ void split_bf16(float x, uint32_t& hi, uint32_t& lo) {
  hi = f32_to_bf16_bits(x);
  lo = f32_to_bf16_bits(x - bf16_bits_to_f32(hi));
}

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
  // bf16 queries: q_out holds each rotated value rounded to bf16 (hi) and q_out_lo the
  // rounded remainder bf16(x - hi) (lo), so hi + lo carries 16 significant bits
  void* q_out_lo;
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
  const void* q;              // rotated queries [n_layers][batch][rows][Hq][D]: bf16 hi for bf16 caches, else fp32
  const void* q_lo;           // bf16 caches: the queries' bf16 lo parts, same layout (null for fp32)
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
  int32_t shared_order;       // sequences share leading pages: run equal work items together
  int32_t n_shared_split;     // splits [0, n) of full-attention layers come from the shared-split kernel
  // splits per (layer, sequence, KV head) in the grid: a full-attention layer's item i is
  // split n_shared_split + i, a windowed layer's split i
  int32_t n_split_grid;
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
  const uint16_t* q;          // rotated queries, bf16 hi parts [n_layers][batch][chunk][Hq][D]
  const uint16_t* q_lo;       // their bf16 lo parts, same layout
  float* out;                 // [n_layers][batch][chunk][Hq][D]
  // attention over pages every sequence shares: partials (reference, sum, unnormalised O)
  // of the rows' splits, for a combine kernel; null in a plain prefill
  float* part_acc;            // [n_layers][batch][chunk][Hq][n_split_max][D]
  float* part_ml;             // [n_layers][batch][chunk][Hq][n_split_max][2]
  float scale_log2;
  int32_t Hq, Hkv, D, group;
  int32_t layer0, n_layers, batch, chunk, max_pages, max_ctx_len, n_qt;
  int32_t n_split_max;
  int32_t n_shared_split, shared_keys;   // shared-split mode: splits [0, n) of shared_keys keys
  int32_t key_lo, part_slot;  // per-sequence mode: keys from key_lo on, partial in this slot
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

// Split-K plan of a row that sees keys [lo, n_keys): splits of kSplit keys from lo on
// (split s = keys [lo + kSplit s, lo + kSplit (s + 1))), a function of the row's own
// length and window only.  Full attention (lo = 0) splits at multiples of kSplit.
__device__ __forceinline__ int split_count(int n_keys, int lo) { return (n_keys - lo + kSplit - 1) / kSplit; }

}  // namespace kvg
