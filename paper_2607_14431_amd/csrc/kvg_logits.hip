// Synthetic logit head over hidden vectors, and the comparison of two logit sets.
//
// The exactness verdict is taken on logits: SHA-256 equality of their bytes (Eq. 1), and as
// corollaries a zero KL divergence between the two softmax distributions and equal argmax
// (Eq. 2); the model's logits pass through a soft cap (Sec. 4.2).  The head here is
//   logits[r][v] = cap * tanh(z / cap),  z = sum_k bf16(hidden[r][k]) * W[v][k]
// (z itself when cap = 0), fp32 accumulation, W bf16 [V][H].
//
// Head kernel: the contraction runs on v_mfma_f32_32x32x16_bf16 with A = 32 vocabulary rows
// of W and B = 32 hidden rows, so a decode batch of up to 32 rows reads W exactly once; W
// streams from HBM and bounds the kernel.  Both operands are in the fragment-major packing
// (kvg_logits.h): W packed once by kvg_logits_pack, the hidden rows converted to bf16 and
// packed into the workspace by each call.  Lane (r, h) of fragment t of 64-element block kb
// holds row r and elements 64 kb + 32 h + 8 t .. + 8, for both operands, so the MFMA sums
// every element of the block exactly once, and each fragment load of a wave is 1 KiB of
// consecutive bytes: a wave streams each of its four 32-row blocks of W as one sequential
// run of H * 64 bytes.  A wave owns 128 vocabulary rows (four accumulators sharing each B
// fragment) and keeps two blocks in flight.  Hidden rows past the input are zero; vocabulary
// blocks past the padded end re-read the last block and are not stored.
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

__device__ __forceinline__ uint4 ld16(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }
// W is streamed once per launch (nontemporal loads): one row 372 -> 337 us, 50 rows
// 448 -> 428 us at 262,144 x 4,096.
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_stream(const uint16_t* p) {
  const u32x4v v = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

// Position of packed 16-byte unit u: matrix row and first element (see packed_unit).
struct UnitPos {
  int64_t row, k;
};
__device__ __forceinline__ UnitPos unit_pos(int64_t u, int n_kb) {
  const int lane = (int)(u & 63);
  const int t = (int)((u >> 6) & 3);
  const int m = (int)((u >> 8) & 3);
  const int64_t rest = u >> 10;
  const int64_t kb = rest % n_kb, blk = rest / n_kb;
  return {kPackRows * blk + 32 * m + (lane & 31), 64 * kb + 32 * (lane >> 5) + 8 * t};
}

// hidden fp32 [rows][H] -> packed bf16, nearest-even; padding rows are zero
__global__ __launch_bounds__(kThreads) void hidden_pack_kernel(const LogitArgs a) {
  const int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (u >= (int64_t)a.rows_pad * a.H / 8) return;
  const UnitPos p = unit_pos(u, a.H / 64);
  uint4 o = make_uint4(0, 0, 0, 0);
  if (p.row < a.rows) {
    const float* src = a.hidden + p.row * a.H + p.k;
    const float4 x0 = *reinterpret_cast<const float4*>(src);
    const float4 x1 = *reinterpret_cast<const float4*>(src + 4);
    const f32x8 x = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    o = __builtin_bit_cast(uint4, __builtin_convertvector(x, bf16x8));
  }
  *reinterpret_cast<uint4*>(a.hidden_packed + u * 8) = o;
}

// W bf16 [V][H] row-major -> packed; rows past V are zero
__global__ __launch_bounds__(kThreads) void weight_pack_kernel(const PackArgs a) {
  const int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (u >= packed_rows(a.V) * a.H / 8) return;
  const UnitPos p = unit_pos(u, a.H / 64);
  const uint4 o = p.row < a.V ? ld16(a.w + p.row * a.H + p.k) : make_uint4(0, 0, 0, 0);
  *reinterpret_cast<uint4*>(a.packed + u * 8) = o;
}

// A wave owns MB 32-row blocks of the vocabulary and NB 32-row tiles of hidden rows: MB x NB
// = 4 accumulators.  MB = 4, NB = 1 serves up to 32 hidden rows (a decode batch) with one
// read of W; MB = 2, NB = 2 and MB = 1, NB = 4 serve up to 64 and 128 rows per read.
template <int MB, int NB>
struct Frags {
  uint4 w[MB][4];    // [vocab block][fragment]
  uint4 h[NB][4];    // [row tile][fragment]
};

template <int MB, int NB>
__global__ __launch_bounds__(kThreads) void logit_head_kernel(const LogitArgs a) {
  constexpr int kWaveVocab = 32 * MB;
  constexpr int kGroupVocab = 4 * kWaveVocab;
  constexpr int kRows = 32 * NB;
  const int n_vt = (a.V + kGroupVocab - 1) / kGroupVocab;
  const int vt = blockIdx.x % n_vt;
  const int nt = blockIdx.x / n_vt;              // group of kRows hidden rows
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 31, lh = lane >> 5;
  const int v0 = vt * kGroupVocab + wave * kWaveVocab;
  if (v0 >= a.V) return;                         // no barrier below: a whole wave may leave
  const int r0 = nt * kRows;

  const int nk = a.H / 64;
  const int last_b32 = (int)(packed_rows(a.V) / 32) - 1;   // padded blocks hold zeros
  const uint16_t* wblk[MB];
  const uint16_t* hblk[NB];
#pragma unroll
  for (int m = 0; m < MB; ++m) wblk[m] = a.w_packed + packed_unit(min(v0 / 32 + m, last_b32), 0, 0, lane, nk) * 8;
#pragma unroll
  for (int n = 0; n < NB; ++n) hblk[n] = a.hidden_packed + packed_unit(r0 / 32 + n, 0, 0, lane, nk) * 8;

  // step kb of a 128-row block starts 16 units of 64 lanes (16 KiB) after step kb - 1
  auto load = [&](int kb, Frags<MB, NB>& f) {
    const int64_t off = (int64_t)kb * 16 * 64 * 8;
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int t = 0; t < 4; ++t) f.w[m][t] = ld16_stream(wblk[m] + off + t * 64 * 8);
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int t = 0; t < 4; ++t) f.h[n][t] = ld16(hblk[n] + off + t * 64 * 8);
  };
  f32x16 acc[MB][NB];
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[m][n][q] = 0.0f;
  auto compute = [&](const Frags<MB, NB>& f) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int n = 0; n < NB; ++n)
          acc[m][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(f.w[m][t]), as_bf16x8(f.h[n][t]),
                                                              acc[m][n], 0, 0, 0);
  };

  // H is a multiple of 128, so steps come in pairs; every load is unconditional (the last
  // one re-reads the final step), which keeps the next step's loads in flight across the
  // loop's back edge.  The scheduling barriers keep each step's loads where they are
  // issued here (the scheduler would otherwise sink them towards their use).
  Frags<MB, NB> x, y;
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

  // lane (r, h) holds, in accumulator element q of (m, n), hidden row r0 + 32 n + r and
  // vocabulary row v0 + 32 m + 8 (q / 4) + 4 h + q % 4
  const bool vec = (a.V & 3) == 0;
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    const int row = r0 + 32 * n + lr;
    if (row >= a.rows) continue;
    float* orow = a.out + (int64_t)row * a.V;
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int v = v0 + 32 * m + 8 * q4 + 4 * lh;
        float l[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float z = acc[m][n][4 * q4 + e];
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

template <int MB, int NB>
void launch_head(const LogitArgs& a, hipStream_t stream) {
  const int64_t n_vt = (a.V + 128 * MB - 1) / (128 * MB);
  const int64_t n_nt = (a.rows + 32 * NB - 1) / (32 * NB);
  logit_head_kernel<MB, NB><<<dim3((unsigned)(n_vt * n_nt)), kThreads, 0, stream>>>(a);
}

hipError_t launch_logits(const LogitArgs& a, hipStream_t stream) {
  const int64_t n8 = (int64_t)a.rows_pad * a.H / 8;
  hidden_pack_kernel<<<dim3((unsigned)((n8 + kThreads - 1) / kThreads)), kThreads, 0, stream>>>(a);
  if (a.rows <= 32)
    launch_head<4, 1>(a, stream);
  else if (a.rows <= 64)
    launch_head<2, 2>(a, stream);
  else
    launch_head<1, 4>(a, stream);
  return hipGetLastError();
}

hipError_t launch_logits_pack(const PackArgs& a, hipStream_t stream) {
  const int64_t n8 = packed_rows(a.V) * a.H / 8;
  weight_pack_kernel<<<dim3((unsigned)((n8 + kThreads - 1) / kThreads)), kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_logit_compare(const CompareArgs& c, hipStream_t stream) {
  logit_compare_kernel<<<dim3((unsigned)c.rows), kThreads, 0, stream>>>(c);
  return hipGetLastError();
}

}  // namespace kvg
