// GPU side of the seeded input generator (the numpy side is synth/philox.py).
//
// Philox4x32-10 (Salmon et al., SC'11) with counter (index lo, index hi, stream lo,
// stream hi) and key (seed lo, seed hi); twelve 10-bit uniforms summed minus 6138
// (Irwin-Hall(12), an integer in [-6138, 6138]); value = z * 2^(sigma_log2 - 10), exact in
// fp32; bf16 storage rounds that value to nearest even.  Generates inputs only.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int64_t kTokenStride = 1LL << 26;

__device__ __forceinline__ void philox_round(uint32_t c[4], uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t hi0 = __umulhi(M0, c[0]), lo0 = M0 * c[0];
  const uint32_t hi1 = __umulhi(M1, c[2]), lo1 = M1 * c[2];
  const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
  c[0] = n0;
  c[1] = lo1;
  c[2] = n2;
  c[3] = lo0;
}

__device__ __forceinline__ int32_t irwin_hall12(uint64_t index, uint64_t stream, uint64_t seed) {
  uint32_t c[4] = {(uint32_t)index, (uint32_t)(index >> 32), (uint32_t)stream, (uint32_t)(stream >> 32)};
  uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    philox_round(c, k0, k1);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  int32_t s = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) s += (int32_t)(c[j] & 1023u) + (int32_t)((c[j] >> 10) & 1023u) + (int32_t)((c[j] >> 20) & 1023u);
  return s - 6138;
}

struct FillArgs {
  void* dst;
  int64_t layer_stride;     // elements between consecutive layers in dst
  int64_t n_per_layer;      // n_tokens * H * D
  int64_t layer_id0;
  int64_t t0;               // token offset inside the stream
  int64_t hd;               // H * D
  uint64_t seed, stream;
  int32_t n_layers, sigma_log2, bf16;
};

__global__ __launch_bounds__(256) void fill_kernel(const FillArgs a) {
  const int64_t n = a.n_per_layer * a.n_layers;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t l = e / a.n_per_layer;
    const int64_t r = e - l * a.n_per_layer;      // (t * H + h) * D + d
    const uint64_t index = (uint64_t)(((a.layer_id0 + l) * kTokenStride + a.t0) * a.hd + r);
    const int32_t z = irwin_hall12(index, a.stream, a.seed);
    const float v = ldexpf((float)z, a.sigma_log2 - 10);
    const int64_t off = l * a.layer_stride + r;
    if (a.bf16) {
      uint32_t u = __float_as_uint(v);
      u += 0x7FFFu + ((u >> 16) & 1u);
      reinterpret_cast<uint16_t*>(a.dst)[off] = (uint16_t)(u >> 16);
    } else {
      reinterpret_cast<float*>(a.dst)[off] = v;
    }
  }
}

}  // namespace

extern "C" {

// Fill dst[l * layer_stride + (t * H + h) * D + d] for l < n_layers, t < n_tokens with the
// value of element ((layer_id0 + l) * 2^26 + t0 + t) * H * D + h * D + d of the stream.
// Returns 0 on success, a HIP error code otherwise.
int synth_fill(void* dst, int64_t layer_stride, int32_t n_layers, int64_t layer_id0, int64_t t0,
               int64_t n_tokens, int32_t n_heads, int32_t head_dim, uint64_t seed, uint64_t stream,
               int32_t sigma_log2, int32_t bf16, void* hip_stream) {
  if (dst == nullptr || n_layers <= 0 || n_tokens <= 0 || n_heads <= 0 || head_dim <= 0) return -1;
  FillArgs a;
  a.dst = dst;
  a.layer_stride = layer_stride;
  a.hd = (int64_t)n_heads * head_dim;
  a.n_per_layer = n_tokens * a.hd;
  a.layer_id0 = layer_id0;
  a.t0 = t0;
  a.seed = seed;
  a.stream = stream;
  a.n_layers = n_layers;
  a.sigma_log2 = sigma_log2;
  a.bf16 = bf16;
  const int64_t n = a.n_per_layer * n_layers;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  fill_kernel<<<dim3((unsigned)blocks), 256, 0, static_cast<hipStream_t>(hip_stream)>>>(a);
  return (int)hipGetLastError();
}

}  // extern "C"
