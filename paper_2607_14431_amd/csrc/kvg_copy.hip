// Deposit (gather) and graft (scatter) of a block's pages.
//
// The payload is [L][2 (K, V)][n_block_pages][Hkv][P][D]; one page of one layer and one
// of K/V is a contiguous chunk of page_bytes on both sides (64 KiB for the 12B-class
// geometry).  Each workgroup moves one 4 KiB slice of one chunk, one 16-byte vector per
// lane, so a wavefront touches 1 KiB of consecutive bytes per instruction and the launch
// has hundreds of thousands of small workgroups: on MI355X this shape streams faster than
// fewer workgroups that each move a whole page (measured with a copy sweep).  Rows at or
// beyond n_tokens in the block's last page are written as zeros by the deposit and left
// untouched by the graft.
//
// A relocated graft is one launch: per (layer, page) the first workgroups re-rotate the
// page's keys (each lane a vector at element e0 of a row and its partner at e0 + D/2 with half
// pairing, or the pairs inside one vector when interleaved, with the per-call (cos, sin)
// table of d * theta_i) and the following ones copy its values, so rotation and plain copy
// workgroups of neighbouring pages share the CUs and the launch has a single tail.
#include "kvg_device.h"
#include "kvg_launch.h"

namespace kvg {

namespace {

constexpr int kThreads = 256;
constexpr int kSliceVec = kThreads;    // 16-byte vectors per workgroup slice (4 KiB)

// Every byte is read once and written once, so both sides are streaming (nontemporal)
// accesses: measured on the 12B-class block, the deposit (random pages -> contiguous
// payload) runs 8% faster and the graft 1% faster than with default cache policy.
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16(const void* p) {
  const u32x4v v = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st16(void* p, const uint4& v) {
  const u32x4v t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, reinterpret_cast<u32x4v*>(p));
}

// Workgroup -> (layer, kv, logical page p, slice); `kinds` = 2 covers K and V, 1 covers one.
struct Slice {
  int l, kv, p, slice;
};

__device__ __forceinline__ Slice slice_of(const CopyArgs& a, int slices_per_page, int kinds) {
  int64_t w = blockIdx.x;
  Slice s;
  s.slice = (int)(w % slices_per_page);
  w /= slices_per_page;
  s.p = (int)(w % a.n_block_pages);
  w /= a.n_block_pages;
  s.kv = (int)(w % kinds);
  s.l = (int)(w / kinds);
  return s;
}

__device__ __forceinline__ int slices_per_page(const CopyArgs& a) {
  return (int)((a.page_bytes / 16 + kSliceVec - 1) / kSliceVec);
}

__global__ __launch_bounds__(kThreads) void deposit_kernel(const CopyArgs a) {
  const Slice s = slice_of(a, slices_per_page(a), 2);
  const int nvec = (int)(a.page_bytes >> 4);
  const int idx = s.slice * kSliceVec + threadIdx.x;
  if (idx >= nvec) return;
  const int32_t page = a.block_table[a.first_page + s.p];
  const bool ok = page >= 0 && page < a.n_pages;
  const int rows = min(kPage, a.n_tokens - s.p * kPage);
  const int r = (idx / (a.row_bytes >> 4)) % kPage;
  const char* pool = reinterpret_cast<const char*>(s.kv ? a.v_pool : a.k_pool) + (int64_t)s.l * a.layer_bytes;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (ok && r < rows) v = ld16(pool + (int64_t)page * a.page_bytes + ((int64_t)idx << 4));
  char* dst = reinterpret_cast<char*>(a.payload) + (((int64_t)s.l * 2 + s.kv) * a.n_block_pages + s.p) * a.page_bytes;
  st16(dst + ((int64_t)idx << 4), v);
}

// One 16-byte vector of a page: rows past the block's last valid row are left untouched.
__device__ __forceinline__ void graft_vector(const CopyArgs& a, int l, int kv, int p, int32_t page, int idx) {
  const int rows = min(kPage, a.n_tokens - p * kPage);
  const int r = (idx / (a.row_bytes >> 4)) % kPage;
  if (r >= rows) return;
  const char* src = reinterpret_cast<const char*>(a.payload) +
                    (((int64_t)l * 2 + kv) * a.n_block_pages + p) * a.page_bytes;
  char* pool = reinterpret_cast<char*>(kv ? a.v_pool : a.k_pool) + (int64_t)l * a.layer_bytes +
               (int64_t)page * a.page_bytes;
  st16(pool + ((int64_t)idx << 4), ld16(src + ((int64_t)idx << 4)));
}

// Plain scatter: the own-position graft (K and V).
__global__ __launch_bounds__(kThreads) void graft_kernel(const CopyArgs a) {
  const Slice s = slice_of(a, slices_per_page(a), 2);
  const int idx = s.slice * kSliceVec + threadIdx.x;
  if (idx >= (int)(a.page_bytes >> 4)) return;
  const int32_t page = a.block_table[a.first_page + s.p];
  if (page < 0 || page >= a.n_pages) return;
  graft_vector(a, s.l, s.kv, s.p, page, idx);
}

// The rotation of E consecutive stored values (one vector) with their partners: x[e] pairs
// with y[e] (half pairing: y is the vector D/2 further) or x[2i] with x[2i + 1] (interleaved),
// pair index pi0 + e (half) or pi0 + e / 2 (interleaved).  bf16 rows are unpacked with shifts
// and repacked two at a time with v_cvt_pk_bf16_f32 (round to nearest even, finite values);
// other types go through their element accessors.
template <typename T, bool kHalf>
__device__ __forceinline__ void rotate_vectors(uint4& va, uint4& vb, int pi0, const float* cs) {
  constexpr int E = Elem<T>::kPerVec;
  if constexpr (sizeof(T) == 2) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      uint32_t& wa = (&va.x)[w];
      uint32_t& wb = (&vb.x)[w];
      float x0 = __uint_as_float(wa << 16), x1 = __uint_as_float(wa & 0xFFFF0000u);
      if constexpr (kHalf) {
        float y0 = __uint_as_float(wb << 16), y1 = __uint_as_float(wb & 0xFFFF0000u);
        rotate_pair(x0, y0, cs[2 * (pi0 + 2 * w)], cs[2 * (pi0 + 2 * w) + 1]);
        rotate_pair(x1, y1, cs[2 * (pi0 + 2 * w + 1)], cs[2 * (pi0 + 2 * w + 1) + 1]);
        wb = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){y0, y1}, bf16x2_t));
      } else {
        rotate_pair(x0, x1, cs[2 * (pi0 + w)], cs[2 * (pi0 + w) + 1]);
      }
      wa = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){x0, x1}, bf16x2_t));
    }
  } else if constexpr (kHalf) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float x = Elem<T>::get(va, e), y = Elem<T>::get(vb, e);
      rotate_pair(x, y, cs[2 * (pi0 + e)], cs[2 * (pi0 + e) + 1]);
      Elem<T>::put(va, e, x);
      Elem<T>::put(vb, e, y);
    }
  } else {
#pragma unroll
    for (int e = 0; e < E; e += 2) {
      float x = Elem<T>::get(va, e), y = Elem<T>::get(va, e + 1);
      rotate_pair(x, y, cs[2 * (pi0 + e / 2)], cs[2 * (pi0 + e / 2) + 1]);
      Elem<T>::put(va, e, x);
      Elem<T>::put(va, e + 1, y);
    }
  }
}

// Relocated graft, one launch.  Workgroup = (layer, page, slice): slices [0, k_slices) rotate
// the page's keys (one item per lane: a vector, and with half pairing its partner D/2 further),
// slices [k_slices, k_slices + v_slices) copy its values (one vector per lane).
template <typename T>
__global__ __launch_bounds__(kThreads) void graft_relocate_kernel(const CopyArgs a, int items_per_row, int k_slices,
                                                                  int v_slices) {
  constexpr int E = Elem<T>::kPerVec;
  const int per_page = k_slices + v_slices;
  const int slice = blockIdx.x % per_page;
  const int p = (blockIdx.x / per_page) % a.n_block_pages;
  const int l = blockIdx.x / per_page / a.n_block_pages;
  const int32_t page = a.block_table[a.first_page + p];
  if (page < 0 || page >= a.n_pages) return;
  if (slice >= k_slices) {
    const int idx = (slice - k_slices) * kSliceVec + threadIdx.x;
    if (idx < (int)(a.page_bytes >> 4)) graft_vector(a, l, 1, p, page, idx);
    return;
  }
  const int it = slice * kThreads + threadIdx.x;
  if (it >= a.Hkv * kPage * items_per_row) return;
  const int rows = min(kPage, a.n_tokens - p * kPage);
  const int rowid = it / items_per_row;            // h * P + r
  if (rowid % kPage >= rows) return;
  const T* src = reinterpret_cast<const T*>(reinterpret_cast<const char*>(a.payload) +
                                            (((int64_t)l * 2) * a.n_block_pages + p) * a.page_bytes);
  T* dst = reinterpret_cast<T*>(reinterpret_cast<char*>(a.k_pool) + (int64_t)l * a.layer_bytes +
                                (int64_t)page * a.page_bytes);
  const int D = a.D, half = D >> 1;
  const int e0 = (it - rowid * items_per_row) * E;
  const int64_t off = (int64_t)rowid * D + e0;
  if (a.pairing == 0) {
    uint4 va = ld16(src + off), vb = ld16(src + off + half);
    rotate_vectors<T, true>(va, vb, e0, a.cs);
    st16(dst + off, va);
    st16(dst + off + half, vb);
  } else {
    uint4 va = ld16(src + off), vb = va;
    rotate_vectors<T, false>(va, vb, e0 / 2, a.cs);
    st16(dst + off, va);
  }
}

int host_slices(const CopyArgs& a) { return (int)((a.page_bytes / 16 + kSliceVec - 1) / kSliceVec); }

}  // namespace

hipError_t launch_deposit(const CopyArgs& a, hipStream_t stream) {
  const int64_t n_wg = (int64_t)a.n_layers * 2 * a.n_block_pages * host_slices(a);
  deposit_kernel<<<dim3((unsigned)n_wg), kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

int64_t copy_workgroups(const CopyArgs& a, int dtype) {
  if (!a.relocate) return (int64_t)a.n_layers * 2 * a.n_block_pages * host_slices(a);
  const int E = dtype == kDtypeFp8 ? 16 : dtype == kDtypeBf16 ? 8 : 4;
  const int items_per_row = a.pairing == 0 ? (a.D / 2) / E : a.D / E;
  const int k_slices = (a.Hkv * kPage * items_per_row + kThreads - 1) / kThreads;
  return (int64_t)a.n_layers * a.n_block_pages * (k_slices + host_slices(a));
}

hipError_t launch_graft(const CopyArgs& a, int dtype, hipStream_t stream) {
  if (!a.relocate) {
    graft_kernel<<<dim3((unsigned)copy_workgroups(a, dtype)), kThreads, 0, stream>>>(a);
    return hipGetLastError();
  }
  const int E = dtype == kDtypeFp8 ? 16 : dtype == kDtypeBf16 ? 8 : 4;
  const int items_per_row = a.pairing == 0 ? (a.D / 2) / E : a.D / E;
  const int k_slices = (a.Hkv * kPage * items_per_row + kThreads - 1) / kThreads;
  const int v_slices = host_slices(a);
  const dim3 grid((unsigned)copy_workgroups(a, dtype));
  switch (dtype) {
    case kDtypeF32:
      graft_relocate_kernel<float><<<grid, kThreads, 0, stream>>>(a, items_per_row, k_slices, v_slices);
      break;
    case kDtypeBf16:
      graft_relocate_kernel<uint16_t><<<grid, kThreads, 0, stream>>>(a, items_per_row, k_slices, v_slices);
      break;
    case kDtypeFp8:
      graft_relocate_kernel<uint8_t><<<grid, kThreads, 0, stream>>>(a, items_per_row, k_slices, v_slices);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kvg
