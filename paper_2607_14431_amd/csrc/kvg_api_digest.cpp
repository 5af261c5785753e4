// C ABI of the content digests (declarations and contracts in include/kvg.h).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>

#include "kvg.h"
#include "kvg_digest.h"

namespace {

int digest_hip_status(hipError_t e) { return e == hipSuccess ? KVG_OK : KVG_E_HIP; }

uint64_t pow2_at_least(uint64_t n) {
  uint64_t p = 64;
  while (p < n) p <<= 1;
  return p;
}

constexpr size_t kAlign = 256;

size_t align_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

// Merkle workspace: two ping-pong levels of ceil(n / 2) digests each.
size_t merkle_ws(uint64_t n_leaves) { return 2 * align_up((size_t)((n_leaves + 1) / 2) * 32); }

size_t dedup_ws(uint64_t n_leaves) {
  const uint64_t slots = pow2_at_least(2 * n_leaves);
  return 2 * align_up((size_t)slots * sizeof(unsigned long long));
}

// Element bytes of a storage dtype code, 0 for an unknown code.
size_t dtype_bytes(int32_t dtype) {
  return dtype == KVG_F32 ? 4 : dtype == KVG_BF16 ? 2 : dtype == KVG_FP8_E4M3 ? 1 : 0;
}

// Leaf bytes of a header's digest (one page of one KV head), 0 when the geometry is invalid
// or the payload size does not follow from it.
uint32_t header_leaf_bytes(const kvg_artifact_hdr* h) {
  if (h == nullptr || h->magic != KVG_ARTIFACT_MAGIC || h->version != KVG_ARTIFACT_VERSION) return 0;
  const size_t e = dtype_bytes(h->dtype);
  if (e == 0 || h->n_layers <= 0 || h->n_kv_heads <= 0 || h->head_dim <= 0 || h->page_size <= 0 || h->n_tokens <= 0)
    return 0;
  const uint64_t leaf = (uint64_t)h->page_size * h->head_dim * e;
  const uint64_t pages = ((uint64_t)h->n_tokens + h->page_size - 1) / h->page_size;
  if (leaf % 64 != 0 || leaf > UINT32_MAX) return 0;
  if (h->payload_bytes != (uint64_t)h->n_layers * 2 * pages * h->n_kv_heads * leaf) return 0;
  return (uint32_t)leaf;
}

struct ArtifactWs {
  size_t digests, merkle, root, total;
};

ArtifactWs artifact_ws(uint64_t n_leaves) {
  ArtifactWs w;
  w.digests = align_up((size_t)n_leaves * 32);
  w.merkle = merkle_ws(n_leaves);
  w.root = align_up(32);
  w.total = w.digests + w.merkle + w.root;
  return w;
}

// The payload's Merkle root over leaf_bytes leaves, computed on `stream` and copied to the
// host (the call waits for the stream).
int payload_root(const void* payload, uint64_t n_bytes, uint32_t leaf_bytes, void* ws, size_t ws_bytes,
                 hipStream_t stream, uint8_t* root_host) {
  if (payload == nullptr || ws == nullptr) return KVG_E_INVAL;
  if (reinterpret_cast<uintptr_t>(payload) % 16 != 0 || reinterpret_cast<uintptr_t>(ws) % 16 != 0) return KVG_E_ALIGN;
  const uint64_t n_leaves = (n_bytes + leaf_bytes - 1) / leaf_bytes;
  const ArtifactWs w = artifact_ws(n_leaves);
  if (ws_bytes < w.total) return KVG_E_WORKSPACE;
  uint8_t* digests = static_cast<uint8_t*>(ws);
  uint8_t* merkle = digests + w.digests;
  uint8_t* root = merkle + w.merkle;
  int st = kvg_leaf_digests(payload, n_bytes, leaf_bytes, digests, stream);
  if (st != KVG_OK) return st;
  st = kvg_merkle_root(digests, n_leaves, root, merkle, w.merkle, stream);
  if (st != KVG_OK) return st;
  if (hipMemcpyAsync(root_host, root, 32, hipMemcpyDeviceToHost, stream) != hipSuccess) return KVG_E_HIP;
  return digest_hip_status(hipStreamSynchronize(stream));
}

}  // namespace

extern "C" {

size_t kvg_artifact_digest_workspace_bytes(const kvg_artifact_hdr* hdr) {
  const uint32_t leaf = header_leaf_bytes(hdr);
  if (leaf == 0) return 0;
  return artifact_ws((hdr->payload_bytes + leaf - 1) / leaf).total;
}

int kvg_artifact_seal(kvg_artifact_hdr* hdr, const void* payload, void* ws_dev, size_t ws_bytes, void* stream) {
  if (hdr == nullptr || payload == nullptr) return KVG_E_INVAL;
  const uint32_t leaf = header_leaf_bytes(hdr);
  if (leaf == 0) return KVG_E_CORRUPT;
  uint8_t root[32];
  const int st = payload_root(payload, hdr->payload_bytes, leaf, ws_dev, ws_bytes, static_cast<hipStream_t>(stream),
                              root);
  if (st != KVG_OK) return st;
  std::memcpy(hdr->digest, root, 32);
  hdr->digest_leaf_bytes = leaf;
  return KVG_OK;
}

int kvg_artifact_verify(const kvg_artifact_hdr* hdr, const void* payload, void* ws_dev, size_t ws_bytes,
                        void* stream) {
  if (hdr == nullptr || payload == nullptr) return KVG_E_INVAL;
  const uint32_t leaf = header_leaf_bytes(hdr);
  if (leaf == 0 || hdr->digest_leaf_bytes != leaf) return KVG_E_CORRUPT;
  uint8_t root[32];
  const int st = payload_root(payload, hdr->payload_bytes, leaf, ws_dev, ws_bytes, static_cast<hipStream_t>(stream),
                              root);
  if (st != KVG_OK) return st;
  return std::memcmp(root, hdr->digest, 32) == 0 ? KVG_OK : KVG_E_CORRUPT;
}

int kvg_leaf_digests(const void* data_dev, uint64_t n_bytes, uint32_t leaf_bytes, uint8_t* digests_dev,
                     void* stream) {
  if (data_dev == nullptr || digests_dev == nullptr || n_bytes == 0 || leaf_bytes == 0 || leaf_bytes % 64 != 0)
    return KVG_E_INVAL;
  if (reinterpret_cast<uintptr_t>(data_dev) % 16 != 0 || reinterpret_cast<uintptr_t>(digests_dev) % 16 != 0)
    return KVG_E_ALIGN;
  kvg::DigestArgs a;
  a.data = data_dev;
  a.n_bytes = n_bytes;
  a.leaf_bytes = leaf_bytes;
  a.n_leaves = (n_bytes + leaf_bytes - 1) / leaf_bytes;
  a.out = digests_dev;
  return digest_hip_status(kvg::launch_leaf_digests(a, static_cast<hipStream_t>(stream)));
}

size_t kvg_merkle_workspace_bytes(uint64_t n_leaves) { return n_leaves == 0 ? 0 : merkle_ws(n_leaves); }

int kvg_merkle_root(const uint8_t* digests_dev, uint64_t n_leaves, uint8_t* root_dev, void* ws_dev, size_t ws_bytes,
                    void* stream) {
  if (digests_dev == nullptr || root_dev == nullptr || n_leaves == 0) return KVG_E_INVAL;
  if (reinterpret_cast<uintptr_t>(digests_dev) % 16 != 0 || reinterpret_cast<uintptr_t>(root_dev) % 16 != 0)
    return KVG_E_ALIGN;
  if (ws_dev == nullptr || ws_bytes < merkle_ws(n_leaves)) return KVG_E_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws_dev) % 16 != 0) return KVG_E_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* buf[2] = {static_cast<uint8_t*>(ws_dev),
                     static_cast<uint8_t*>(ws_dev) + align_up((size_t)((n_leaves + 1) / 2) * 32)};
  const uint8_t* src = digests_dev;
  uint64_t n = n_leaves;
  int which = 0;
  do {
    const uint64_t n_out = (n + 1) / 2;
    uint8_t* dst = (n_out == 1) ? root_dev : buf[which];
    const hipError_t e = kvg::launch_merkle_level(src, n, dst, s);
    if (e != hipSuccess) return KVG_E_HIP;
    src = dst;
    n = n_out;
    which ^= 1;
  } while (n > 1);
  return KVG_OK;
}

size_t kvg_dedup_workspace_bytes(uint64_t n_leaves) { return n_leaves == 0 ? 0 : dedup_ws(n_leaves); }

int kvg_dedup_map(const uint8_t* digests_dev, uint64_t n_leaves, int64_t* first_index_dev, int32_t* n_unresolved_dev,
                  void* ws_dev, size_t ws_bytes, void* stream) {
  if (digests_dev == nullptr || first_index_dev == nullptr || n_unresolved_dev == nullptr || n_leaves == 0)
    return KVG_E_INVAL;
  if (reinterpret_cast<uintptr_t>(digests_dev) % 16 != 0) return KVG_E_ALIGN;
  if (ws_dev == nullptr || ws_bytes < dedup_ws(n_leaves)) return KVG_E_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws_dev) % 8 != 0) return KVG_E_ALIGN;
  const uint64_t slots = pow2_at_least(2 * n_leaves);
  kvg::DedupArgs a;
  a.digests = digests_dev;
  a.n_leaves = n_leaves;
  a.keys = static_cast<unsigned long long*>(ws_dev);
  a.first = reinterpret_cast<unsigned long long*>(static_cast<uint8_t*>(ws_dev) +
                                                  align_up((size_t)slots * sizeof(unsigned long long)));
  a.table_slots = slots;
  a.first_index = first_index_dev;
  a.n_unresolved = n_unresolved_dev;
  return digest_hip_status(kvg::launch_dedup(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
