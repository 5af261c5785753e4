// Synthetic logit head over hidden vectors, and the comparison of two logit sets.
//
// The exactness verdict is taken on logits: SHA-256 equality of their bytes (Eq. 1), and as
// corollaries a zero KL divergence between the two softmax distributions and equal argmax
// (Eq. 2); the model's logits pass through a soft cap (Sec. 4.2).  The head here is
//   logits[r][v] = cap * tanh(z / cap),  z = sum_k bf16(hidden[r][k]) * W[v][k]
// (z itself when cap = 0), fp32 accumulation, W bf16 [V][H].
//
// Head kernel: the contraction runs on v_mfma_f32_32x32x16_bf16 with A = 32 vocabulary rows
// of W and B = 32 hidden rows (bf16, converted once into the workspace), so a decode batch of
// up to 32 rows reads W exactly once; W streams from HBM and bounds the kernel.  A wave owns
// 128 vocabulary rows (four accumulators sharing each B fragment) and walks the hidden
// dimension in 64-element blocks, two blocks in flight: lane (r, h) of the wave loads the 64
// contiguous bytes [64 h, 64 h + 64) of the block's 128 bytes of its rows, as four 16-byte
// fragments.  The MFMA k index of fragment t is matched to hidden element 32 h + 8 t + e of
// the block for both operands, so every element of the block is summed exactly once.
// Hidden rows past the input are zero in the workspace; vocabulary rows past V re-read row
// V - 1 and are not stored.
//
// Compare kernel: one workgroup per row: first-index argmax of each logit vector, the log-sum-
// exp of each and KL(softmax(a) || softmax(b)) = sum_i p_i ((a_i - b_i) - (lse_a - lse_b)),
// in fp64 with fixed-order reductions, so byte-equal inputs give exactly 0.
#include "kvg_logits.h"

#include <math.h>

namespace kvg {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kWaveVocab = 128;                  // vocabulary rows per wave
constexpr int kGroupVocab = 4 * kWaveVocab;      // per workgroup of four waves

__device__ __forceinline__ uint4 ld16(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

// hidden fp32 [rows][H] -> bf16 [rows_pad][H], nearest-even; padding rows are zero
__global__ __launch_bounds__(kThreads) void hidden_to_bf16_kernel(const LogitArgs a) {
  const int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 8;   // first of 8 elements
  if (i >= (int64_t)a.rows_pad * a.H) return;
  const int64_t r = i / a.H;
  uint4 o = make_uint4(0, 0, 0, 0);
  if (r < a.rows) {
    const float4 x0 = *reinterpret_cast<const float4*>(a.hidden + i);
    const float4 x1 = *reinterpret_cast<const float4*>(a.hidden + i + 4);
    const f32x8 x = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    o = __builtin_bit_cast(uint4, __builtin_convertvector(x, bf16x8));
  }
  *reinterpret_cast<uint4*>(a.hidden_bf16 + i) = o;
}

struct Frags {
  uint4 w[4][4];     // [vocab block][fragment]
  uint4 h[4];        // [fragment]
};

__global__ __launch_bounds__(kThreads) void logit_head_kernel(const LogitArgs a) {
  const int n_vt = (a.V + kGroupVocab - 1) / kGroupVocab;
  const int vt = blockIdx.x % n_vt;
  const int nt = blockIdx.x / n_vt;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 31, lh = lane >> 5;
  const int v0 = vt * kGroupVocab + wave * kWaveVocab;
  if (v0 >= a.V) return;                         // no barrier below: a whole wave may leave
  const int r0 = nt * kLogitRowTile;

  const uint16_t* wrow[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) wrow[m] = a.w + (int64_t)min(v0 + 32 * m + lr, a.V - 1) * a.H + lh * 32;
  const uint16_t* hrow = a.hidden_bf16 + (int64_t)(r0 + lr) * a.H + lh * 32;

  auto load = [&](int kb, Frags& f) {
    const int64_t off = (int64_t)kb * 64;
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int t = 0; t < 4; ++t) f.w[m][t] = ld16(wrow[m] + off + 8 * t);
#pragma unroll
    for (int t = 0; t < 4; ++t) f.h[t] = ld16(hrow + off + 8 * t);
  };
  f32x16 acc[4];
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[m][q] = 0.0f;
  auto compute = [&](const Frags& f) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int m = 0; m < 4; ++m)
        acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(f.w[m][t]), as_bf16x8(f.h[t]), acc[m], 0, 0, 0);
  };

  // H is a multiple of 128, so blocks come in pairs; every load is unconditional (the last
  // one re-reads the final block), which keeps the next block's loads in flight across the
  // loop's back edge.  The scheduling barriers keep each block's loads where they are
  // issued here (the scheduler would otherwise sink them towards their use).
  const int nk = a.H / 64;
  Frags x, y;
  load(0, x);
  for (int kb = 0; kb < nk; kb += 2) {
    load(kb + 1, y);
    __builtin_amdgcn_sched_barrier(0);
    compute(x);
    __builtin_amdgcn_sched_barrier(0);
    load(min(kb + 2, nk - 1), x);
    __builtin_amdgcn_sched_barrier(0);
    compute(y);
    __builtin_amdgcn_sched_barrier(0);
  }

  // lane (r, h) holds hidden row r0 + r and, in accumulator element q of block m, vocabulary
  // row v0 + 32 m + 8 (q / 4) + 4 h + q % 4
  const int row = r0 + lr;
  if (row >= a.rows) return;
  float* orow = a.out + (int64_t)row * a.V;
  const bool vec = (a.V & 3) == 0;
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int v = v0 + 32 * m + 8 * q4 + 4 * lh;
      float l[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float z = acc[m][4 * q4 + e];
        l[e] = a.cap > 0.0f ? a.cap * tanhf(z / a.cap) : z;
      }
      if (vec && v + 3 < a.V) {
        *reinterpret_cast<float4*>(orow + v) = make_float4(l[0], l[1], l[2], l[3]);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (v + e < a.V) orow[v + e] = l[e];
      }
    }
}

// ---------------------------------------------------------------------------- comparison
struct ArgMax {
  float v;
  int i;
};

// the larger value; of equal values the smaller index (the first maximum)
__device__ __forceinline__ ArgMax better(ArgMax x, ArgMax y) {
  return (y.v > x.v || (y.v == x.v && y.i < x.i)) ? y : x;
}

__device__ __forceinline__ ArgMax block_argmax(ArgMax x, ArgMax* sh) {
  sh[threadIdx.x] = x;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) sh[threadIdx.x] = better(sh[threadIdx.x], sh[threadIdx.x + s]);
    __syncthreads();
  }
  const ArgMax r = sh[0];
  __syncthreads();
  return r;
}

__device__ __forceinline__ double block_sum(double x, double* sh) {
  sh[threadIdx.x] = x;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  const double r = sh[0];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kThreads) void logit_compare_kernel(const CompareArgs c) {
  __shared__ ArgMax sh_arg[kThreads];
  __shared__ double sh_sum[kThreads];
  const int64_t base = (int64_t)blockIdx.x * c.V;
  const float* a = c.a + base;
  const float* b = c.b + base;
  const int tid = threadIdx.x;

  ArgMax ma{-INFINITY, c.V}, mb{-INFINITY, c.V};
  for (int i = tid; i < c.V; i += kThreads) {
    ma = better(ma, ArgMax{a[i], i});
    mb = better(mb, ArgMax{b[i], i});
  }
  ma = block_argmax(ma, sh_arg);
  mb = block_argmax(mb, sh_arg);

  double sa = 0.0, sb = 0.0;
  for (int i = tid; i < c.V; i += kThreads) {
    sa += exp((double)a[i] - (double)ma.v);
    sb += exp((double)b[i] - (double)mb.v);
  }
  sa = block_sum(sa, sh_sum);
  sb = block_sum(sb, sh_sum);
  const double lse_a = (double)ma.v + log(sa);
  const double lse_b = (double)mb.v + log(sb);

  double kl = 0.0;
  for (int i = tid; i < c.V; i += kThreads) {
    const double la = (double)a[i] - lse_a;
    const double lb = (double)b[i] - lse_b;
    kl += exp(la) * (la - lb);
  }
  kl = block_sum(kl, sh_sum);
  if (tid == 0) {
    c.kl[blockIdx.x] = kl;
    c.arg_a[blockIdx.x] = ma.i;
    c.arg_b[blockIdx.x] = mb.i;
  }
}

}  // namespace

hipError_t launch_logits(const LogitArgs& a, hipStream_t stream) {
  const int64_t n8 = (int64_t)a.rows_pad * a.H / 8;
  hidden_to_bf16_kernel<<<dim3((unsigned)((n8 + kThreads - 1) / kThreads)), kThreads, 0, stream>>>(a);
  const int64_t n_vt = (a.V + kGroupVocab - 1) / kGroupVocab;
  const int64_t n_nt = a.rows_pad / kLogitRowTile;
  logit_head_kernel<<<dim3((unsigned)(n_vt * n_nt)), kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_logit_compare(const CompareArgs& c, hipStream_t stream) {
  logit_compare_kernel<<<dim3((unsigned)c.rows), kThreads, 0, stream>>>(c);
  return hipGetLastError();
}

}  // namespace kvg
