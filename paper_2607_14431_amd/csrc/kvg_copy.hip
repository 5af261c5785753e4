// Deposit (gather) and graft (scatter) of a block's pages.
//
// The payload is [L][2 (K, V)][n_block_pages][Hkv][P][D]; one page of one layer and one
// of K/V is a contiguous chunk of page_bytes on both sides (64 KiB for the 12B-class
// geometry), so each workgroup moves one such chunk with 16-byte accesses: every lane
// issues all of its loads before its stores, and a wavefront touches 1 KiB of
// consecutive bytes per instruction.  Rows at or beyond n_tokens in the block's last page
// are written as zeros by the deposit and left untouched by the graft.
//
// A relocated graft re-rotates keys: each lane handles a vector at element e0 of a row
// and its partner at e0 + D/2 (half pairing) or the pairs inside one vector
// (interleaved), rotating with the per-call (cos, sin) table of d * theta_i.
#include "kvg_device.h"
#include "kvg_launch.h"

namespace kvg {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxVecPerThread = 16;   // 64 KiB per pass: 256 lanes * 16 vectors * 16 B

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st16(void* p, const uint4& v) { *reinterpret_cast<uint4*>(p) = v; }

// Chunk for (layer, kv, logical page p) in the pool (via the block table) and the payload.
struct ChunkPtrs {
  char* pool;
  char* payload;
  int rows;        // valid rows in this page
  bool ok;
};

__device__ __forceinline__ ChunkPtrs chunk_ptrs(const CopyArgs& a) {
  const int p = blockIdx.x >> 1;
  const int kv = blockIdx.x & 1;
  const int l = blockIdx.y;
  ChunkPtrs c;
  const int32_t page = a.block_table[a.first_page + p];
  c.ok = page >= 0 && page < a.n_pages;
  char* base = reinterpret_cast<char*>(kv ? a.v_pool : a.k_pool);
  c.pool = base + (int64_t)l * a.layer_bytes + (int64_t)(c.ok ? page : 0) * a.page_bytes;
  c.payload = reinterpret_cast<char*>(a.payload) +
              (((int64_t)l * 2 + kv) * a.n_block_pages + p) * a.page_bytes;
  c.rows = min(kPage, a.n_tokens - p * kPage);
  return c;
}

__global__ __launch_bounds__(kThreads) void deposit_kernel(const CopyArgs a) {
  const ChunkPtrs c = chunk_ptrs(a);
  const int nvec = (int)(a.page_bytes >> 4);
  const int vec_per_row = a.row_bytes >> 4;
  for (int base = 0; base < nvec; base += kThreads * kMaxVecPerThread) {
    uint4 v[kMaxVecPerThread];
#pragma unroll
    for (int j = 0; j < kMaxVecPerThread; ++j) {
      const int idx = base + threadIdx.x + j * kThreads;
      const int r = (idx / vec_per_row) % kPage;
      v[j] = make_uint4(0, 0, 0, 0);
      if (idx < nvec && r < c.rows && c.ok) v[j] = ld16(c.pool + ((int64_t)idx << 4));
    }
#pragma unroll
    for (int j = 0; j < kMaxVecPerThread; ++j) {
      const int idx = base + threadIdx.x + j * kThreads;
      if (idx < nvec) st16(c.payload + ((int64_t)idx << 4), v[j]);
    }
  }
}

// Plain scatter of one chunk; rows at or beyond `rows` are not written.
__device__ __forceinline__ void scatter_chunk(const char* src, char* dst, int nvec, int vec_per_row, int rows) {
  for (int base = 0; base < nvec; base += kThreads * kMaxVecPerThread) {
    uint4 v[kMaxVecPerThread];
#pragma unroll
    for (int j = 0; j < kMaxVecPerThread; ++j) {
      const int idx = base + threadIdx.x + j * kThreads;
      if (idx < nvec) v[j] = ld16(src + ((int64_t)idx << 4));
    }
#pragma unroll
    for (int j = 0; j < kMaxVecPerThread; ++j) {
      const int idx = base + threadIdx.x + j * kThreads;
      const int r = (idx / vec_per_row) % kPage;
      if (idx < nvec && r < rows) st16(dst + ((int64_t)idx << 4), v[j]);
    }
  }
}

__global__ __launch_bounds__(kThreads) void graft_kernel(const CopyArgs a) {
  const ChunkPtrs c = chunk_ptrs(a);
  if (!c.ok) return;
  scatter_chunk(c.payload, c.pool, (int)(a.page_bytes >> 4), a.row_bytes >> 4, c.rows);
}

// Relocated graft, key chunks: rotate by the call's (cos, sin) table.  Value chunks go
// through graft_v_kernel, launched right after on the same stream.
template <typename T>
__global__ __launch_bounds__(kThreads) void graft_relocate_k_kernel(const CopyArgs a) {
  constexpr int E = Elem<T>::kPerVec;
  const int p = blockIdx.x;
  const int l = blockIdx.y;
  const int32_t page = a.block_table[a.first_page + p];
  if (page < 0 || page >= a.n_pages) return;
  const int rows = min(kPage, a.n_tokens - p * kPage);
  const T* src = reinterpret_cast<const T*>(reinterpret_cast<const char*>(a.payload) +
                                            (((int64_t)l * 2) * a.n_block_pages + p) * a.page_bytes);
  T* dst = reinterpret_cast<T*>(reinterpret_cast<char*>(a.k_pool) + (int64_t)l * a.layer_bytes +
                                (int64_t)page * a.page_bytes);
  const int D = a.D, half = D >> 1;
  const int items_per_row = (a.pairing == 0) ? (half / E) : (D / E);
  const int n_items = a.Hkv * kPage * items_per_row;
  for (int it = threadIdx.x; it < n_items; it += kThreads) {
    const int rowid = it / items_per_row;            // h * P + r
    const int r = rowid % kPage;
    if (r >= rows) continue;
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
}

// Value chunks of a relocated graft: the plain scatter restricted to kv = 1.
__global__ __launch_bounds__(kThreads) void graft_v_kernel(const CopyArgs a) {
  const int p = blockIdx.x;
  const int l = blockIdx.y;
  const int32_t page = a.block_table[a.first_page + p];
  if (page < 0 || page >= a.n_pages) return;
  const int rows = min(kPage, a.n_tokens - p * kPage);
  const char* src = reinterpret_cast<const char*>(a.payload) + (((int64_t)l * 2 + 1) * a.n_block_pages + p) * a.page_bytes;
  char* dst = reinterpret_cast<char*>(a.v_pool) + (int64_t)l * a.layer_bytes + (int64_t)page * a.page_bytes;
  scatter_chunk(src, dst, (int)(a.page_bytes >> 4), a.row_bytes >> 4, rows);
}

}  // namespace

hipError_t launch_deposit(const CopyArgs& a, hipStream_t stream) {
  const dim3 grid(2 * a.n_block_pages, a.n_layers);
  deposit_kernel<<<grid, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_graft(const CopyArgs& a, int bf16, hipStream_t stream) {
  if (!a.relocate) {
    const dim3 grid(2 * a.n_block_pages, a.n_layers);
    graft_kernel<<<grid, kThreads, 0, stream>>>(a);
    return hipGetLastError();
  }
  const dim3 grid(a.n_block_pages, a.n_layers);
  if (bf16)
    graft_relocate_k_kernel<uint16_t><<<grid, kThreads, 0, stream>>>(a);
  else
    graft_relocate_k_kernel<float><<<grid, kThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  graft_v_kernel<<<grid, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace kvg
