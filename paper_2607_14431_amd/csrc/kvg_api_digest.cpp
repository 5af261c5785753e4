// C ABI of the content digests (declarations and contracts in include/kvg.h).
#include <hip/hip_runtime.h>

#include <cstdint>

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

}  // namespace

extern "C" {

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
