// Kernel arguments and launchers of the content digests (SHA-256 leaves, Merkle levels,
// dedup table).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace kvg {

struct DigestArgs {
  const void* data;            // 16-byte aligned device buffer
  uint64_t n_bytes;
  uint32_t leaf_bytes;         // positive multiple of 64
  uint64_t n_leaves;           // ceil(n_bytes / leaf_bytes)
  uint8_t* out;                // [n_leaves][32]
};

struct DedupArgs {
  const uint8_t* digests;      // [n_leaves][32], 16-byte aligned
  uint64_t n_leaves;
  unsigned long long* keys;    // [table_slots] first 8 digest bytes, or all ones when empty
  unsigned long long* first;   // [table_slots] smallest leaf index per key
  uint64_t table_slots;        // power of two, >= 2 * n_leaves
  int64_t* first_index;        // [n_leaves] output
  int32_t* n_unresolved;       // [1] output
};

hipError_t launch_leaf_digests(const DigestArgs& a, hipStream_t stream);
hipError_t launch_merkle_level(const uint8_t* in, uint64_t n_in, uint8_t* out, hipStream_t stream);
hipError_t launch_dedup(const DedupArgs& a, hipStream_t stream);

}  // namespace kvg
