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
// A relocated graft re-rotates keys: each lane handles a vector at element e0 of a row and
// its partner at e0 + D/2 (half pairing) or the pairs inside one vector (interleaved),
// rotating with the per-call (cos, sin) table of d * theta_i.
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

// Plain scatter: the own-position graft (kinds = 2, K and V) and the values of a relocated
// graft (kinds = 1, V only).
__global__ __launch_bounds__(kThreads) void graft_kernel(const CopyArgs a, int kinds) {
  const Slice s = slice_of(a, slices_per_page(a), kinds);
  const int kv = kinds == 2 ? s.kv : 1;
  const int nvec = (int)(a.page_bytes >> 4);
  const int idx = s.slice * kSliceVec + threadIdx.x;
  if (idx >= nvec) return;
  const int32_t page = a.block_table[a.first_page + s.p];
  if (page < 0 || page >= a.n_pages) return;
  const int rows = min(kPage, a.n_tokens - s.p * kPage);
  const int r = (idx / (a.row_bytes >> 4)) % kPage;
  if (r >= rows) return;
  const char* src = reinterpret_cast<const char*>(a.payload) +
                    (((int64_t)s.l * 2 + kv) * a.n_block_pages + s.p) * a.page_bytes;
  char* pool = reinterpret_cast<char*>(kv ? a.v_pool : a.k_pool) + (int64_t)s.l * a.layer_bytes +
               (int64_t)page * a.page_bytes;
  st16(pool + ((int64_t)idx << 4), ld16(src + ((int64_t)idx << 4)));
}

// Relocated graft, key chunks: rotate by the call's (cos, sin) table.  One item = one
// 16-byte vector (interleaved) or a vector and its partner D/2 further (half pairing).
template <typename T>
__global__ __launch_bounds__(kThreads) void graft_relocate_k_kernel(const CopyArgs a, int items_per_row,
                                                                    int slices) {
  constexpr int E = Elem<T>::kPerVec;
  const int slice = blockIdx.x % slices;
  const int p = (blockIdx.x / slices) % a.n_block_pages;
  const int l = blockIdx.x / slices / a.n_block_pages;
  const int it = slice * kThreads + threadIdx.x;
  if (it >= a.Hkv * kPage * items_per_row) return;
  const int32_t page = a.block_table[a.first_page + p];
  if (page < 0 || page >= a.n_pages) return;
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
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float x = Elem<T>::get(va, e), y = Elem<T>::get(vb, e);
      const int pi = e0 + e;
      rotate_pair(x, y, a.cs[2 * pi], a.cs[2 * pi + 1]);
      Elem<T>::put(va, e, x);
      Elem<T>::put(vb, e, y);
    }
    st16(dst + off, va);
    st16(dst + off + half, vb);
  } else {
    uint4 va = ld16(src + off);
#pragma unroll
    for (int e = 0; e < E; e += 2) {
      float x = Elem<T>::get(va, e), y = Elem<T>::get(va, e + 1);
      const int pi = (e0 + e) >> 1;
      rotate_pair(x, y, a.cs[2 * pi], a.cs[2 * pi + 1]);
      Elem<T>::put(va, e, x);
      Elem<T>::put(va, e + 1, y);
    }
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

hipError_t launch_graft(const CopyArgs& a, int dtype, hipStream_t stream) {
  if (!a.relocate) {
    const int64_t n_wg = (int64_t)a.n_layers * 2 * a.n_block_pages * host_slices(a);
    graft_kernel<<<dim3((unsigned)n_wg), kThreads, 0, stream>>>(a, 2);
    return hipGetLastError();
  }
  const int E = dtype == kDtypeFp8 ? 16 : dtype == kDtypeBf16 ? 8 : 4;
  const int items_per_row = a.pairing == 0 ? (a.D / 2) / E : a.D / E;
  const int slices = (a.Hkv * kPage * items_per_row + kThreads - 1) / kThreads;
  const int64_t n_wg_k = (int64_t)a.n_layers * a.n_block_pages * slices;
  switch (dtype) {
    case kDtypeF32:
      graft_relocate_k_kernel<float><<<dim3((unsigned)n_wg_k), kThreads, 0, stream>>>(a, items_per_row, slices);
      break;
    case kDtypeBf16:
      graft_relocate_k_kernel<uint16_t><<<dim3((unsigned)n_wg_k), kThreads, 0, stream>>>(a, items_per_row, slices);
      break;
    case kDtypeFp8:
      graft_relocate_k_kernel<uint8_t><<<dim3((unsigned)n_wg_k), kThreads, 0, stream>>>(a, items_per_row, slices);
      break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n_wg_v = (int64_t)a.n_layers * a.n_block_pages * host_slices(a);
  graft_kernel<<<dim3((unsigned)n_wg_v), kThreads, 0, stream>>>(a, 1);
  return hipGetLastError();
}

}  // namespace kvg
