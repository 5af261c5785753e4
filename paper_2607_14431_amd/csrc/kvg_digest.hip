// SHA-256 (FIPS 180-4) content digests of device buffers: one lane per leaf, one launch
// per Merkle-tree level, and a content-addressed dedup table.
//
// Leaves are independent messages, so a wavefront hashes 64 leaves side by side; each
// lane walks its leaf in 64-byte blocks (four 16-byte loads, big-endian words by byte
// permute) through the 64-round compression in registers.  The work is integer ALU:
// rotations are v_alignbit, the message schedule lives in a 16-word register ring.
#include "kvg_digest.h"

#include <climits>

namespace kvg {

namespace {

// ---- constants from their definitions (FIPS 180-4, 4.2.2 and 5.3.3): the first 32 bits
// of the fractional parts of the cube roots of the first 64 primes (round constants) and of
// the square roots of the first 8 primes (initial hash value), by exact integer roots.
typedef unsigned __int128 u128;

constexpr u128 iroot(u128 n, int k, u128 hi) {
  u128 lo = 0;
  while (lo < hi) {
    const u128 m = (lo + hi + 1) / 2;
    const u128 p = (k == 3) ? m * m * m : m * m;
    if (p <= n) lo = m;
    else hi = m - 1;
  }
  return lo;
}

struct Sha256Consts {
  uint32_t k[64];
  uint32_t h0[8];
};

constexpr Sha256Consts make_sha256_consts() {
  Sha256Consts c{};
  int n = 0;
  for (uint32_t p = 2; n < 64; ++p) {
    bool prime = true;
    for (uint32_t d = 2; d * d <= p; ++d)
      if (p % d == 0) {
        prime = false;
        break;
      }
    if (!prime) continue;
    // floor(cbrt(p) * 2^32) = floor(cbrt(p * 2^96)); keeping the low 32 bits drops the
    // integer part.  cbrt(311 * 2^96) < 2^36, so cubes stay below 2^108.
    c.k[n] = (uint32_t)iroot((u128)p << 96, 3, (u128)1 << 36);
    if (n < 8) c.h0[n] = (uint32_t)iroot((u128)p << 64, 2, (u128)1 << 35);
    ++n;
  }
  return c;
}

constexpr Sha256Consts kSha = make_sha256_consts();
static_assert(kSha.h0[0] == 0x6a09e667u && kSha.k[0] == 0x428a2f98u && kSha.k[63] == 0xc67178f2u,
              "SHA-256 constants");

__device__ __forceinline__ uint32_t rotr(uint32_t x, int n) { return __builtin_amdgcn_alignbit(x, x, n); }
__device__ __forceinline__ uint32_t be32(uint32_t x) { return __builtin_bswap32(x); }
// a ^ b ^ c in one v_bitop3_b32.  The truth table's bit (x << 2 | y << 1 | z) is the result
// for operand bits x, y, z: 0x96 = parity, 0xCA = x ? y : z, 0xE8 = majority.
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// One compression of block w (big-endian words; the ring is overwritten) into state st.
__device__ __forceinline__ void compress(uint32_t (&st)[8], uint32_t (&w)[16]) {
  uint32_t a = st[0], b = st[1], c = st[2], d = st[3], e = st[4], f = st[5], g = st[6], h = st[7];
#pragma unroll
  for (int t = 0; t < 64; ++t) {
    uint32_t wt;
    if (t < 16) {
      wt = w[t];
    } else {
      const uint32_t w15 = w[(t - 15) & 15], w2 = w[(t - 2) & 15];
      const uint32_t s0 = xor3(rotr(w15, 7), rotr(w15, 18), w15 >> 3);
      const uint32_t s1 = xor3(rotr(w2, 17), rotr(w2, 19), w2 >> 10);
      wt = w[t & 15] + s0 + w[(t - 7) & 15] + s1;          // W[t-16] + s0 + W[t-7] + s1
      w[t & 15] = wt;
    }
    const uint32_t big_s1 = xor3(rotr(e, 6), rotr(e, 11), rotr(e, 25));
    const uint32_t ch = __builtin_amdgcn_bitop3_b32(e, f, g, 0xCA);     // e ? f : g
    const uint32_t t1 = h + big_s1 + ch + kSha.k[t] + wt;
    const uint32_t big_s0 = xor3(rotr(a, 2), rotr(a, 13), rotr(a, 22));
    const uint32_t maj = __builtin_amdgcn_bitop3_b32(a, b, c, 0xE8);    // majority of a, b, c
    const uint32_t t2 = big_s0 + maj;
    h = g;
    g = f;
    f = e;
    e = d + t1;
    d = c;
    c = b;
    b = a;
    a = t1 + t2;
  }
  st[0] += a;
  st[1] += b;
  st[2] += c;
  st[3] += d;
  st[4] += e;
  st[5] += f;
  st[6] += g;
  st[7] += h;
}

__device__ __forceinline__ void init_state(uint32_t (&st)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) st[i] = kSha.h0[i];
}

// digest words -> 32 bytes, big-endian
__device__ __forceinline__ void store_digest(uint8_t* out, const uint32_t (&st)[8]) {
  uint4* o = reinterpret_cast<uint4*>(out);
  o[0] = make_uint4(be32(st[0]), be32(st[1]), be32(st[2]), be32(st[3]));
  o[1] = make_uint4(be32(st[4]), be32(st[5]), be32(st[6]), be32(st[7]));
}

__device__ __forceinline__ void load_digest_words(const uint8_t* p, uint32_t (&w)[8]) {
  const uint4 a = reinterpret_cast<const uint4*>(p)[0], b = reinterpret_cast<const uint4*>(p)[1];
  w[0] = be32(a.x);
  w[1] = be32(a.y);
  w[2] = be32(a.z);
  w[3] = be32(a.w);
  w[4] = be32(b.x);
  w[5] = be32(b.y);
  w[6] = be32(b.z);
  w[7] = be32(b.w);
}

constexpr int kDigestThreads = 256;

// SHA-256 of leaf i = bytes [i * leaf_bytes, min((i + 1) * leaf_bytes, n_bytes)).
__global__ __launch_bounds__(kDigestThreads) void leaf_sha256_kernel(const DigestArgs a) {
  const uint64_t leaf = (uint64_t)blockIdx.x * kDigestThreads + threadIdx.x;
  if (leaf >= a.n_leaves) return;
  const uint64_t off = leaf * a.leaf_bytes;
  const uint64_t len = min((uint64_t)a.leaf_bytes, a.n_bytes - off);
  const uint64_t n_full = len / 64;
  const uint8_t* base = reinterpret_cast<const uint8_t*>(a.data) + off;
  const uint4* p = reinterpret_cast<const uint4*>(base);

  uint32_t st[8];
  init_state(st);
  for (uint64_t blk = 0; blk < n_full; ++blk) {
    uint32_t w[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 v = p[blk * 4 + q];
      w[4 * q + 0] = be32(v.x);
      w[4 * q + 1] = be32(v.y);
      w[4 * q + 2] = be32(v.z);
      w[4 * q + 3] = be32(v.w);
    }
    compress(st, w);
  }
  // padding: the remaining bytes, 0x80, zeros, then the bit length in the last 8 bytes;
  // a second block when fewer than 9 bytes are left in the first
  const uint32_t rem = (uint32_t)(len - n_full * 64);
  const uint8_t* tail = base + n_full * 64;
  uint32_t w[16];
  if (rem == 0) {                    // every leaf but a ragged last one
    w[0] = 0x80u << 24;
#pragma unroll
    for (int j = 1; j < 16; ++j) w[j] = 0;
  } else {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      uint32_t word = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const uint32_t i = 4 * j + b;
        uint32_t byte = 0;
        if (i < rem) byte = tail[i];                 // only bytes inside the leaf are read
        else if (i == rem) byte = 0x80u;
        word |= byte << (24 - 8 * b);
      }
      w[j] = word;
    }
  }
  const uint64_t bits = len * 8;
  if (rem >= 56) {
    compress(st, w);
#pragma unroll
    for (int i = 0; i < 16; ++i) w[i] = 0;
  }
  w[14] = (uint32_t)(bits >> 32);
  w[15] = (uint32_t)bits;
  compress(st, w);
  store_digest(a.out + leaf * 32, st);
}

// One tree level: node i = SHA-256(0x01 || in[2i] || in[2i+1]), or in[2i] moved up when it
// is the level's odd last node.  The 65-byte message spans two blocks.
__global__ __launch_bounds__(kDigestThreads) void merkle_level_kernel(const uint8_t* in, uint64_t n_in,
                                                                       uint8_t* out) {
  const uint64_t i = (uint64_t)blockIdx.x * kDigestThreads + threadIdx.x;
  const uint64_t n_out = (n_in + 1) / 2;
  if (i >= n_out) return;
  if (2 * i + 1 >= n_in) {
    reinterpret_cast<uint4*>(out + i * 32)[0] = reinterpret_cast<const uint4*>(in + 2 * i * 32)[0];
    reinterpret_cast<uint4*>(out + i * 32)[1] = reinterpret_cast<const uint4*>(in + 2 * i * 32)[1];
    return;
  }
  uint32_t l[8], r[8];
  load_digest_words(in + 2 * i * 32, l);
  load_digest_words(in + (2 * i + 1) * 32, r);
  uint32_t st[8];
  init_state(st);
  uint32_t w[16];
  // message bytes m[0] = 0x01, m[1..32] = left, m[33..64] = right; word j = m[4j..4j+3]
  w[0] = (0x01u << 24) | (l[0] >> 8);
#pragma unroll
  for (int j = 1; j < 8; ++j) w[j] = (l[j - 1] << 24) | (l[j] >> 8);
  w[8] = (l[7] << 24) | (r[0] >> 8);
#pragma unroll
  for (int j = 9; j < 16; ++j) w[j] = (r[j - 9] << 24) | (r[j - 8] >> 8);
  compress(st, w);
  w[0] = (r[7] << 24) | (0x80u << 16);
#pragma unroll
  for (int j = 1; j < 15; ++j) w[j] = 0;
  w[15] = 65 * 8;
  compress(st, w);
  store_digest(out + i * 32, st);
}

// ---- dedup: open addressing keyed by the first 8 digest bytes
constexpr unsigned long long kEmpty = ~0ull;

__device__ __forceinline__ unsigned long long dedup_key(const uint8_t* d) {
  const unsigned long long k = reinterpret_cast<const unsigned long long*>(d)[0];
  return k == kEmpty ? kEmpty - 1 : k;                // the empty marker is never a key
}

__global__ __launch_bounds__(kDigestThreads) void dedup_clear_kernel(const DedupArgs a) {
  const uint64_t s = (uint64_t)blockIdx.x * kDigestThreads + threadIdx.x;
  if (s < a.table_slots) {
    a.keys[s] = kEmpty;
    a.first[s] = (unsigned long long)INT64_MAX;
  }
  if (s == 0) a.n_unresolved[0] = 0;
}

// Every leaf claims (or finds) its key's slot and lowers the slot's smallest index.  The
// table has at least twice as many slots as leaves, so every probe sequence ends.
__global__ __launch_bounds__(kDigestThreads) void dedup_insert_kernel(const DedupArgs a) {
  const uint64_t i = (uint64_t)blockIdx.x * kDigestThreads + threadIdx.x;
  if (i >= a.n_leaves) return;
  const unsigned long long k = dedup_key(a.digests + i * 32);
  const uint64_t mask = a.table_slots - 1;
  uint64_t s = k & mask;
  for (uint64_t probe = 0; probe < a.table_slots; ++probe) {
    const unsigned long long prev = atomicCAS(&a.keys[s], kEmpty, k);
    if (prev == kEmpty || prev == k) {
      atomicMin(&a.first[s], (unsigned long long)i);
      return;
    }
    s = (s + 1) & mask;
  }
}

// The smallest index recorded under the leaf's key, confirmed on all 32 bytes.
__global__ __launch_bounds__(kDigestThreads) void dedup_resolve_kernel(const DedupArgs a) {
  const uint64_t i = (uint64_t)blockIdx.x * kDigestThreads + threadIdx.x;
  if (i >= a.n_leaves) return;
  const uint8_t* di = a.digests + i * 32;
  const unsigned long long k = dedup_key(di);
  const uint64_t mask = a.table_slots - 1;
  uint64_t s = k & mask;
  int64_t res = -1;
  for (uint64_t probe = 0; probe < a.table_slots; ++probe) {
    const unsigned long long key = a.keys[s];
    if (key == k) {
      const uint64_t rep = a.first[s];
      const uint4* x = reinterpret_cast<const uint4*>(di);
      const uint4* y = reinterpret_cast<const uint4*>(a.digests + rep * 32);
      const uint4 x0 = x[0], x1 = x[1], y0 = y[0], y1 = y[1];
      const bool same = x0.x == y0.x && x0.y == y0.y && x0.z == y0.z && x0.w == y0.w && x1.x == y1.x &&
                        x1.y == y1.y && x1.z == y1.z && x1.w == y1.w;
      res = same ? (int64_t)rep : -1;
      break;
    }
    if (key == kEmpty) break;
    s = (s + 1) & mask;
  }
  a.first_index[i] = res;
  if (res < 0) atomicAdd(a.n_unresolved, 1);
}

inline unsigned grid_for(uint64_t n) { return (unsigned)((n + kDigestThreads - 1) / kDigestThreads); }

}  // namespace

hipError_t launch_leaf_digests(const DigestArgs& a, hipStream_t stream) {
  leaf_sha256_kernel<<<grid_for(a.n_leaves), kDigestThreads, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_merkle_level(const uint8_t* in, uint64_t n_in, uint8_t* out, hipStream_t stream) {
  merkle_level_kernel<<<grid_for((n_in + 1) / 2), kDigestThreads, 0, stream>>>(in, n_in, out);
  return hipGetLastError();
}

hipError_t launch_dedup(const DedupArgs& a, hipStream_t stream) {
  dedup_clear_kernel<<<grid_for(a.table_slots), kDigestThreads, 0, stream>>>(a);
  dedup_insert_kernel<<<grid_for(a.n_leaves), kDigestThreads, 0, stream>>>(a);
  dedup_resolve_kernel<<<grid_for(a.n_leaves), kDigestThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace kvg
