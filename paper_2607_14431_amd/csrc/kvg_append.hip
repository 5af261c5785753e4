// KV-append: fresh computation of new tokens' keys/values into the paged cache, plus the
// rotated queries the attention kernels read.
//
// One workgroup per (sequence, new token) and group of layers.  The token's absolute
// position is the same for every layer and head, so the workgroup computes the D/2
// angles pos * theta_i in fp64 once, takes cos/sin in fp64, rounds them to fp32 into
// LDS, and every thread then rotates 16-byte vectors of its rows with the fixed fp32
// formula of rotate_pair().  Keys are rounded to the storage dtype (nearest even) and
// written through the block table; values are copied (rounded to fp8 for an fp8 cache,
// whose raw inputs are bf16); queries go to the workspace.
#include "kvg_device.h"
#include "kvg_launch.h"

#include <type_traits>

namespace kvg {

namespace {

// Raw rows are read once and cache rows written once: streaming (nontemporal) accesses
// (the 4,096-token 12B-class prefix: 693 -> 670 us).
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16(const void* p) {
  const u32x4v v = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st16(void* p, const uint4& v) {
  const u32x4v t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, reinterpret_cast<u32x4v*>(p));
}

// Rotated pair values of one item: half pairing reads vectors at element offsets e0 and
// e0 + D/2 (E pairs); interleaved reads one vector (E/2 pairs).
template <typename T>
struct RotItem {
  static constexpr int E = Elem<T>::kPerVec;
  float x[2][E];   // [0]: vector at e0, [1]: partner vector (half pairing only)
};

template <typename T>
__device__ __forceinline__ void rotate_item(const T* row, int e0, int half, int pairing,
                                            const float* cs, RotItem<T>& it) {
  constexpr int E = Elem<T>::kPerVec;
  if (pairing == 0) {
    const uint4 va = ld16(row + e0);
    const uint4 vb = ld16(row + e0 + half);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float a = Elem<T>::get(va, e), b = Elem<T>::get(vb, e);
      const int p = e0 + e;
      rotate_pair(a, b, cs[2 * p], cs[2 * p + 1]);
      it.x[0][e] = a;
      it.x[1][e] = b;
    }
  } else {
    const uint4 va = ld16(row + e0);
#pragma unroll
    for (int e = 0; e < E; e += 2) {
      float a = Elem<T>::get(va, e), b = Elem<T>::get(va, e + 1);
      const int p = (e0 + e) >> 1;
      rotate_pair(a, b, cs[2 * p], cs[2 * p + 1]);
      it.x[0][e] = a;
      it.x[0][e + 1] = b;
    }
  }
}

// E consecutive values stored in type T (16 bytes, or 8 for fp8 from a bf16 item)
template <typename T, int E>
__device__ __forceinline__ void store_elems(T* dst, const float* x) {
  uint32_t w[4];
  pack_words<T, E>(x, w);
  if constexpr (E * sizeof(T) == 16)
    st16(dst, make_uint4(w[0], w[1], w[2], w[3]));
  else
    *reinterpret_cast<uint2*>(dst) = make_uint2(w[0], w[1]);
}

// E (8) fp32 values as bf16 hi and lo parts (split_bf16), one 16-byte vector each
template <int E>
__device__ __forceinline__ void store_split(uint16_t* hi, uint16_t* lo, const float* x) {
  static_assert(E == 8, "one 16-byte vector of bf16");
  uint32_t h[E], l[E];
#pragma unroll
  for (int e = 0; e < E; ++e) split_bf16(x[e], h[e], l[e]);
  st16(hi, make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)));
  st16(lo, make_uint4(l[0] | (l[1] << 16), l[2] | (l[3] << 16), l[4] | (l[5] << 16), l[6] | (l[7] << 16)));
}

template <typename T>
__device__ __forceinline__ void store_vec_f32(float* dst, const float* x) {
  constexpr int E = Elem<T>::kPerVec;
#pragma unroll
  for (int e = 0; e < E; e += 4) st16(dst + e, make_uint4(__float_as_uint(x[e]), __float_as_uint(x[e + 1]),
                                                           __float_as_uint(x[e + 2]), __float_as_uint(x[e + 3])));
}

template <typename T>
__global__ __launch_bounds__(256) void append_kernel(const AppendArgs a) {
  using R = typename RawOf<T>::type;                     // raw input type
  constexpr int E = Elem<R>::kPerVec;                    // elements per item vector
  const int tok = blockIdx.x;
  const int b = tok / a.chunk;
  const int i = tok - b * a.chunk;
  const int ctx = a.ctx_lens[b];
  if (ctx < 0 || ctx > a.max_ctx_len) return;           // uniform: bad metadata, skip
  const int t = ctx + i;                                 // < max_pages * kPage (host check)
  const int32_t page = a.block_tables[(int64_t)b * a.max_pages + t / kPage];
  const bool page_ok = page >= 0 && page < a.n_pages;
  const int64_t pos = a.start_pos[b] + t;
  const int D = a.D, half = D >> 1;

  __shared__ float cs[2 * kMaxHalfDim];
  for (int p = threadIdx.x; p < half; p += blockDim.x) {
    double s, c;
    sincos((double)pos * a.theta[p], &s, &c);
    cs[2 * p] = (float)c;
    cs[2 * p + 1] = (float)s;
  }
  __syncthreads();

  const int items_per_row = (a.pairing == 0) ? (half / E) : (D / E);
  const int vec_per_row = D / E;
  const int l_begin = blockIdx.y * a.layers_per_block;
  const int l_end = min(l_begin + a.layers_per_block, a.n_layers);
  const int row = t % kPage;

  for (int l = l_begin; l < l_end; ++l) {
    const int64_t raw_tok = ((int64_t)l * a.batch + b) * a.chunk + i;
    const int64_t lbase = (int64_t)(a.layer0 + l) * a.layer_elems;
    T* kpool = reinterpret_cast<T*>(a.k_pool) + lbase;
    T* vpool = reinterpret_cast<T*>(a.v_pool) + lbase;
    const R* kraw = reinterpret_cast<const R*>(a.k_raw) + raw_tok * a.Hkv * D;
    const R* vraw = reinterpret_cast<const R*>(a.v_raw) + raw_tok * a.Hkv * D;

    if (page_ok) {
      // keys: rotate, round, store through the block table
      for (int it = threadIdx.x; it < a.Hkv * items_per_row; it += blockDim.x) {
        const int h = it / items_per_row;
        const int e0 = (it - h * items_per_row) * E;
        RotItem<R> r;
        rotate_item<R>(kraw + (int64_t)h * D, e0, half, a.pairing, cs, r);
        T* dst = kpool + (((int64_t)page * a.Hkv + h) * kPage + row) * D;
        store_elems<T, E>(dst + e0, r.x[0]);
        if (a.pairing == 0) store_elems<T, E>(dst + e0 + half, r.x[1]);
      }
      // values: copy (rounded to the storage type when it differs from the raw type)
      for (int it = threadIdx.x; it < a.Hkv * vec_per_row; it += blockDim.x) {
        const int h = it / vec_per_row;
        const int e0 = (it - h * vec_per_row) * E;
        T* dst = vpool + (((int64_t)page * a.Hkv + h) * kPage + row) * D + e0;
        const uint4 raw = ld16(vraw + (int64_t)h * D + e0);
        if constexpr (std::is_same<T, R>::value) {
          st16(dst, raw);
        } else {
          float x[E];
#pragma unroll
          for (int e = 0; e < E; ++e) x[e] = Elem<R>::get(raw, e);
          store_elems<T, E>(dst, x);
        }
      }
    }
    if (a.q_raw != nullptr) {
      const R* qraw = reinterpret_cast<const R*>(a.q_raw) + raw_tok * a.Hq * D;
      for (int it = threadIdx.x; it < a.Hq * items_per_row; it += blockDim.x) {
        const int h = it / items_per_row;
        const int e0 = (it - h * items_per_row) * E;
        RotItem<R> r;
        rotate_item<R>(qraw + (int64_t)h * D, e0, half, a.pairing, cs, r);
        const int64_t qoff = (raw_tok * a.Hq + h) * D;
        if constexpr (sizeof(R) == 2) {
          if (a.q_out_bf16) {                      // bf16 hi + lo queries (bf16 and fp8 caches)
            uint16_t* qh = reinterpret_cast<uint16_t*>(a.q_out) + qoff;
            uint16_t* ql = reinterpret_cast<uint16_t*>(a.q_out_lo) + qoff;
            store_split<E>(qh + e0, ql + e0, r.x[0]);
            if (a.pairing == 0) store_split<E>(qh + e0 + half, ql + e0 + half, r.x[1]);
            continue;
          }
        }
        {
          float* q = reinterpret_cast<float*>(a.q_out) + qoff;
          store_vec_f32<R>(q + e0, r.x[0]);
          if (a.pairing == 0) store_vec_f32<R>(q + e0 + half, r.x[1]);
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, int dtype, hipStream_t stream) {
  const dim3 grid(a.batch * a.chunk, (a.n_layers + a.layers_per_block - 1) / a.layers_per_block);
  switch (dtype) {
    case kDtypeF32: append_kernel<float><<<grid, 256, 0, stream>>>(a); break;
    case kDtypeBf16: append_kernel<uint16_t><<<grid, 256, 0, stream>>>(a); break;
    case kDtypeFp8: append_kernel<uint8_t><<<grid, 256, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kvg
