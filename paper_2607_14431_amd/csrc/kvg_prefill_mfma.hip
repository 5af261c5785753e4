// Chunked-prefill attention on bf16 MFMA (gfx950 v_mfma_f32_32x32x16_bf16) over a paged
// cache: the suffix rows attend causally to the cached (e.g. grafted) prefix and to the
// chunk itself.
//
// Workgroup = (layer, sequence, KV head g, q-tile) with NW waves (8 at head_dim <= 128, 4 at
// 256, where a wave's registers allow only one wave per SIMD).  A q-tile holds
// BM = 32 NW / group query rows for each of the `group` query heads that share KV head g, so
// one K/V tile in LDS serves 32 NW (row, head) pairs; wave w owns 32 consecutive rows of one
// head.
//
// Per 64-key tile (tiles start at absolute multiples of 64 of the logical key index, so a
// row's arithmetic does not depend on how the sequence was chunked):
//   staging       the tile's 4 pages of K and of V are split into shares of 16 or 8
//                 rows, one per wave (the first NCH waves when a row has NCH < NW
//                 16-byte chunks), brought from the paged pools straight into LDS with
//                 buffer_load_dwordx4 ... lds (no registers, no ALU), two stages deep: tile
//                 kt + 1 loads while tile kt is computed (at head_dim 256 its loads are
//                 spread over the MFMA steps of the S phases); the page id of tile kt + 2 is
//                 read while tile kt + 1 loads.  Both tiles stay row-major; the 16-byte
//                 chunks of each row are XOR-swizzled so the reads below are free of bank
//                 conflicts, and every LDS address is (per-lane base) XOR (a constant of the
//                 unrolled step) plus an immediate offset.  Keys past the workgroup's last
//                 row read as zeros (the buffer resource ends at the last row in range:
//                 finite values, masked to p = 0 below).
//   S^T = K Q^T   A = K rows from LDS, B = the wave's queries held in registers as bf16
//                 hi and lo parts (two MFMAs per K fragment, so a score is as accurate as
//                 with fp32 queries: rounding the rotated queries to bf16 alone moves
//                 scores of a peaked softmax by ~1e-2 and outputs by a few 1e-2); C = 32
//                 keys x 32 rows, so each lane owns one query row (lane % 32) and 16 of its
//                 keys, the other half in lane ^ 32.  The tile's two 32-key blocks have
//                 their own accumulators; K fragments are read six k-steps ahead at head_dim
//                 256 (one wave per SIMD: nothing else covers an LDS read), two below.
//   softmax       per 32-key block: causal / window mask (key <= row) on diagonal and
//                 window-edge tiles only, running reference / sum per row in fp32 with exp2
//                 (scale folded into one FMA); both halves of a row exchange their block max
//                 and sum with a VALU half swap; the reference moves only when a block max
//                 exceeds it by 2^8, so most blocks leave O alone.  Block 0's softmax runs in
//                 pieces beside block 1's S MFMAs and block 1's beside block 0's P V MFMAs.
//   O^T += V^T P^T  A = V^T fragments read from the row-major V tile with
//                 ds_read_b64_tr_b16 (a 16-lane group addresses four keys x 16 dims and
//                 each lane receives one dim of the four keys), six steps ahead at head_dim
//                 256 and three below, B = P
//                 rounded to bf16 straight from the S^T registers (the key order inside
//                 each 16-key step is the accumulator's own order, used identically for both
//                 operands); C = O^T, one row per lane so the rescale is a per-lane multiply.
// Every MFMA step is a scheduling region of its own (scheduling barriers), holding the step's
// LDS reads, its share of the tile loads and, in the overlapped phases, one piece of the other
// block's softmax.
#include "kvg_device.h"
#include "kvg_launch.h"

#include <limits.h>
#include <math.h>

#include <type_traits>

namespace kvg {

namespace {

// A lane's value and that of lane ^ 32, as (the value in lanes 0-31, the value in lanes
// 32-63): both halves of the wave get the same pair, so a reduction of the two is the same
// bits in both.  A VALU half swap, where a cross-lane shuffle would be an LDS round trip whose
// wait also drains every LDS read issued before it.
__device__ inline float2 halves32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) char lds_char;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i32x2 lds_i32x2;

constexpr int kTileKeys = 64;
// Fourth word of a raw buffer resource on gfx9-family targets (32-bit data format, no
// swizzle): accesses past num_records return zeros instead of touching memory.
constexpr int kBufferWord3 = 0x00020000;
// LDS fragments read ahead of the MFMAs that use them at head_dim 256 (K and Vᵀ streams)
constexpr int kLookK256 = 6;
constexpr int kLookV256 = 6;
constexpr float kRescale = 8.0f;  // lazy-rescale threshold of a row's reference (log2 units)

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

// two fp32 -> packed bf16, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16_rne(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

// LDS tile layout: row r (0..63) of a tile holds its NCH 16-byte chunks at positions
// chunk ^ swizzle(r).  Only r mod 16 matters, and every swizzle is XOR-linear in the row
// bits, so a load share starting at row r0 (a multiple of its power-of-two size) has the
// swizzle of its own rows XOR swizzle(r0).
//   K (read as one chunk of 32 consecutive rows per lane group): r & 15 puts 16 consecutive
//     rows on 16 distinct chunk positions.
//   V (read transposed: four consecutive rows x two or four adjacent chunks per group):
//     {0, 6, 10, 12}[r & 3] keeps four rows apart both over 8 and over 16 chunk positions.
template <int NCH>
struct Swz {
  __device__ static __forceinline__ int k(int r) { return NCH >= 16 ? (r & 15) : (r & 7); }
  __device__ static __forceinline__ int v(int r) {
    return NCH >= 16 ? ((0xCA60 >> (4 * (r & 3))) & 15) : 2 * (r & 3);
  }
};

// fp8 rows (D bytes) are read 8 bytes at a time: K fragments with ds_read_b64, Vᵀ fragments
// with ds_read_b64_tr_b8 (a 16-lane group's eight 16-byte row pieces, each addressed by a
// lane pair, come back transposed: lane j receives byte j of all eight rows).  The swizzles
// keep each read's rows on distinct banks, counting that 128- and 64-byte rows share a
// 256-byte bank line: K over the 16 rows of a lane half, V over the eight keys
// {0..3, 8..11} (+4) of a group.  All are XOR-linear bit fields of the row and only use
// row bits below 4 (K: below 5 / 16 keys apart never collide within a read).
template <int D>
struct SwzFp8 {
  __device__ static __forceinline__ int k(int r) {
    return D == 256 ? (r & 15) : D == 128 ? ((r >> 1) & 7) : ((r >> 2) & 3);
  }
  __device__ static __forceinline__ int v(int r) {
    return D == 256 ? (r & 15) : D == 128 ? (((r >> 1) & 1) | (((r >> 3) & 1) << 1)) : ((r >> 3) & 1);
  }
};

// eight fp8 values (two words) -> eight bf16 values, exactly
__device__ __forceinline__ uint4 widen_fp8x8(uint32_t lo, uint32_t hi) {
  return make_uint4(__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)lo, 1.0f, false)),
                    __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)lo, 1.0f, true)),
                    __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)hi, 1.0f, false)),
                    __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)hi, 1.0f, true)));
}

// T: cache storage (uint16_t bf16, uint8_t fp8 E4M3).  fp8 tiles are staged as bytes (half the
// HBM, DMA and LDS traffic) and widened to bf16 fragments exactly before the MFMAs.
// NW: waves per workgroup (prefill_mfma_waves), 32 query rows each.
template <typename T, int D, int NW, bool kShared>
__global__ __launch_bounds__(64 * NW) void prefill_mfma_kernel(const PrefillArgs a) {
  constexpr bool kFp8 = sizeof(T) == 1;
  constexpr int RB = D * (int)sizeof(T);   // bytes per cache row
  constexpr int NCH = RB / 16;         // 16-byte chunks per row
  constexpr int NS = D / 16;           // MFMA k-steps over head_dim
  constexpr int ND = D / 32;           // 32-wide blocks of head_dim
  constexpr int kTileChunks = kTileKeys * NCH;
  // A tile of one operand is NCH direct loads of 1 KiB; NWL waves share them, each bringing
  // R consecutive rows (a page or half a page).
  constexpr int NWL = NW < NCH ? NW : NCH;
  constexpr int kLoads = NCH / NWL;                // direct loads per lane per array
  constexpr int R = kTileKeys / NWL;               // rows per loading wave
  static_assert(NCH % NWL == 0 && kPage % R == 0, "load shares must tile the pages");
  using SW = typename std::conditional<kFp8, SwzFp8<D>, Swz<NCH>>::type;
  // One LDS object per stage and operand: with the stage a compile-time constant in each
  // half of the unrolled tile loop, the compiler can tell that the tile being read and the
  // tile being loaded (LDS DMA) do not overlap, so reads never wait for the next tile's
  // loads.  The compiler lays the objects out in the order of their names; the V tiles come
  // first, inside the 64 KiB that an LDS instruction's immediate offset reaches, because
  // their transposed reads are four times as many as the K reads (at head_dim 256 the four
  // tiles take 128 KiB, and reads past 64 KiB need an address add each).
  __shared__ __attribute__((aligned(1024))) uint4 sA_V0[kTileChunks];
  __shared__ __attribute__((aligned(1024))) uint4 sA_V1[kTileChunks];
  __shared__ __attribute__((aligned(1024))) uint4 sB_K0[kTileChunks];
  __shared__ __attribute__((aligned(1024))) uint4 sB_K1[kTileChunks];

  // ---- workgroup coordinates: XCD-aware order
  const int nwg = gridDim.x;
  int id = blockIdx.x;
  const int per_xcd = nwg / 8;
  if (id < per_xcd * 8) id = (id % 8) * per_xcd + id / 8;
  const int G = a.group;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int lrow = lane & 31;
  const int half = lane >> 5;
  // Per lane: its query row's visible keys [row_lo, row_n] and whether it has a row at all;
  // per wave: the smallest and largest row_n of its rows and the first key any of them sees;
  // per workgroup: the tiles [kt_begin, n_tiles) it loads, keys [0, n_hi) in range.
  int l, g, h, b = 0, row = 0, split = 0, row_n, row_lo, wave_first, wave_last, wave_lo, mask_lo;
  int n_hi, kt_begin;
  bool row_ok;
  const int32_t* bt;
  if constexpr (!kShared) {
    // (q-tile, KV head, sequence, layer), heavy (late) q-tiles first
    int qt = id % a.n_qt;
    int rest = id / a.n_qt;
    g = rest % a.Hkv;
    rest /= a.Hkv;
    b = rest % a.batch;
    l = rest / a.batch;
    qt = a.n_qt - 1 - qt;
    const int ctx = a.ctx_lens[b];
    if (ctx < 0 || ctx > a.max_ctx_len) return;
    const int BM = 32 * NW / G;
    const int i0 = qt * BM;
    const int h_local = (wave * 32) / BM;
    const int r0 = (wave * 32) % BM;
    h = g * G + h_local;
    row = i0 + r0 + lrow;                               // chunk row of this lane
    row_ok = row < a.chunk;
    row_n = ctx + row;                                  // its logical index: keys [0, row_n]
    wave_first = ctx + i0 + r0;
    wave_last = ctx + min(i0 + r0 + 31, a.chunk - 1);   // last key any row of this wave sees
    n_hi = ctx + min(i0 + BM, a.chunk);                 // keys [0, n_hi) needed by the workgroup
    // sliding window: row i sees keys (i - W, i]; tiles wholly below the workgroup's first
    // row's window are neither loaded nor visited, tiles below this wave's are visited
    // (every wave takes part in the loads) but not computed
    const int W = layer_window(a, l);
    kt_begin = window_start(W, ctx + i0 + 1) / kTileKeys;
    // keys below key_lo (the shared pages, whose part came from the shared-split mode) are
    // not visited on full-attention layers; the floor never passes the workgroup's first row
    // (only a broken shared-pages promise could make it), so the range is never empty
    if (W == 0) kt_begin = max(kt_begin, min(a.key_lo, ctx + i0) / kTileKeys);
    wave_lo = window_start(W, ctx + i0 + r0 + 1);       // first key any row of this wave sees
    row_lo = window_start(W, row_n + 1);                // first key of this lane's row
    mask_lo = window_start(W, ctx + i0 + r0 + 32);      // keys below it are masked for some row
    bt = a.block_tables + (int64_t)b * a.max_pages;
  } else {
    // Shared split: (row block, split, KV head, layer).  The rows are the batch's query rows
    // (a decode: chunk 1; a suffix prefill: the chunk's rows), one per (sequence, chunk row,
    // query head of the group): wave w of row block rb takes head (rb NW + w) mod G of rows
    // 32 ((rb NW + w) / G) + 0..31 of the (sequence, chunk row) list.  The split's keys
    // [shared_keys s, shared_keys (s + 1)) lie in the pages every sequence shares, read
    // through the first sequence's block table.  Layers with a window are left to the
    // per-sequence kernels.
    const int rb = id % a.n_qt;
    int rest = id / a.n_qt;
    split = rest % a.n_shared_split;
    rest /= a.n_shared_split;
    g = rest % a.Hkv;
    l = rest / a.Hkv;
    if (layer_window(a, l) != 0) return;
    const int wi = rb * NW + wave;
    h = g * G + wi % G;
    const int r = 32 * (wi / G) + lrow;                 // this lane's (sequence, chunk row)
    b = r / a.chunk;
    row = r - b * a.chunk;
    const int ctx = b < a.batch ? a.ctx_lens[b] : -1;
    row_ok = ctx >= 0 && ctx <= a.max_ctx_len;
    row_n = row_ok ? ctx + row : -1;                    // keys [0, ctx + row] (a decode: its new token)
    row_lo = 0;
    int lo = row_ok ? row_n : INT_MAX, hi = row_n;
#pragma unroll
    for (int m = 16; m >= 1; m >>= 1) {
      lo = min(lo, __shfl_xor(lo, m));
      hi = max(hi, __shfl_xor(hi, m));
    }
    wave_first = __builtin_amdgcn_readfirstlane(lo);
    wave_last = __builtin_amdgcn_readfirstlane(hi);
    wave_lo = mask_lo = 0;
    n_hi = (split + 1) * a.shared_keys;
    kt_begin = split * (a.shared_keys / kTileKeys);
    bt = a.block_tables;
  }
  const int n_tiles = (n_hi + kTileKeys - 1) / kTileKeys;
  const int last_page = (n_hi - 1) / kPage;

  const int64_t lbase = (int64_t)(a.layer0 + l) * a.layer_elems;
  const T* kpool = reinterpret_cast<const T*>(a.k_pool) + lbase;
  const T* vpool = reinterpret_cast<const T*>(a.v_pool) + lbase;

  // ---- wave w's share of tile kt (w < NWL): tile rows [w R, w R + R), i.e. rows
  // [r0w, r0w + R) of page kt * 4 + w R / 16, clamped to the last needed page.
  // Instruction i of a wave covers slots [64 i, 64 i + 64) of its R rows: row
  // (64 i + lane) / NCH, position (64 i + lane) % NCH, which holds chunk position ^
  // swizzle(tile row).  Both swizzles are XOR-linear in the row bits, w R has no bits in
  // common with the rows inside a share, and a row step of 64 / NCH rows is 1 KiB, so the
  // byte offset in the page slab is r0w RB + 1024 i + (offset of slot lane) XOR 16
  // swizzle(64 i / NCH) XOR 16 swizzle(w R).
  constexpr int kRowsPerLoad = 64 / NCH;
  const int lrow0 = lane / NCH;
  const int r0w = (wave * R) % kPage;
  const uint32_t k_off0 = lrow0 * RB + 16 * ((lane % NCH) ^ SW::k(lrow0) ^ SW::k(wave * R));
  const uint32_t v_off0 = lrow0 * RB + 16 * ((lane % NCH) ^ SW::v(lrow0) ^ SW::v(wave * R));
  auto page_slot = [&](int kt) { return kt * (kTileKeys / kPage) + (wave * R) / kPage; };
  auto page_of_tile = [&](int kt) -> int32_t { return bt[min(page_slot(kt), last_page)]; };
  // The loads go through a buffer resource over the (page, head) slab (wave-uniform base,
  // 32-bit per-lane offsets).  As MUBUF loads they count only in the vector-memory counter, so
  // the LDS reads of the tile being computed wait for exactly their own data (partial
  // lgkmcnt); a global_load_lds is a FLAT instruction that the compiler must assume can touch
  // LDS out of order, and every LDS wait behind it became a full drain that also waited for
  // the next tile's loads.  The resource ends at the last row of the page inside the range:
  // the hardware bounds check turns rows past it (only on the last needed page, or a whole
  // page past the range) into zeros, finite values that the mask weights by p = 0, with no
  // per-lane arithmetic.
  // the resource over operand pool `pool` for the page of tile kt (page id `page`)
  auto tile_rsrc = [&](const T* pool, int kt, int32_t page) {
    page = __builtin_amdgcn_readfirstlane(page);
    page = (page >= 0 && page < a.n_pages) ? page : 0;
    const int64_t poff = ((int64_t)page * a.Hkv + g) * kPage * D;
    // rows of the page in range (uniform: n_hi is the workgroup's)
    const int rows = __builtin_amdgcn_readfirstlane(min(max(n_hi - page_slot(kt) * kPage, 0), kPage));
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(pool + poff), 0, rows * RB, kBufferWord3);
  };
  // loads [j0, j1) of the 2 kLoads of a tile (K and V alternate) into stage DS
  constexpr int kTileLoads = 2 * kLoads;
  constexpr bool kSpreadLoads = NW == 4;     // one wave per SIMD (head_dim 256)
  auto issue = [&](__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv, auto dst_stage, int j0, int j1) {
    if constexpr (NWL < NW) {
      if (wave >= NWL) return;
    }
    constexpr int DS = decltype(dst_stage)::value;
    lds_char* dk = (lds_char*)(lds_void*)&(DS ? sB_K1 : sB_K0)[wave * R * NCH];
    lds_char* dv = (lds_char*)(lds_void*)&(DS ? sA_V1 : sA_V0)[wave * R * NCH];
    const uint32_t share0 = r0w * RB;                        // the share's first row in the slab
#pragma unroll
    for (int j = j0; j < j1; ++j) {
      const int i = j >> 1;
      if (j & 1) {
        const uint32_t ov = share0 + 1024 * i + (v_off0 ^ (16 * SW::v(i * kRowsPerLoad)));
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(dv + 1024 * i), 16, ov, 0, 0, 0);
      } else {
        const uint32_t ok = share0 + 1024 * i + (k_off0 ^ (16 * SW::k(i * kRowsPerLoad)));
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(dk + 1024 * i), 16, ok, 0, 0, 0);
      }
    }
  };

  // ---- queries of this lane's row (B operand of S^T = K Q^T), zeros past the chunk: the
  // bf16 hi parts qf and lo parts ql (each rotated value is hi + lo to 16 significant bits);
  // every K fragment multiplies both, so a score carries the query to fp32-like accuracy
  uint4 qf[NS], ql[NS];
  {
    const int64_t qrow = kShared ? (((int64_t)l * a.batch + (row_ok ? b : 0)) * a.chunk + (row_ok ? row : 0)) * a.Hq + h
                                 : (((int64_t)l * a.batch + b) * a.chunk + (row_ok ? row : 0)) * a.Hq + h;
    const uint16_t* qp = a.q + qrow * D;
    const uint16_t* qlp = a.q_lo + qrow * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      qf[s] = row_ok ? *reinterpret_cast<const uint4*>(qp + (2 * s + half) * 8) : make_uint4(0, 0, 0, 0);
      ql[s] = row_ok ? *reinterpret_cast<const uint4*>(qlp + (2 * s + half) * 8) : make_uint4(0, 0, 0, 0);
    }
  }

  f32x16 o[ND];
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[d][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  // ---- LDS addressing.  Rows are 2D bytes; a constant below 2D XORed into a row address
  // only permutes that row's chunks, which is exactly the swizzle.
  //   K step ss of 32-key block kb: row kb * 32 + lrow, chunk (2 ss + half) ^ swz(lrow)
  //     = ((row base + 16 (half ^ swz)) ^ (32 ss)) + kb * 32 rows.
  //   V^T step (ks, d), rows 16 ks + rr (+ 8): dims 32 d + 16 (m % 2) + 4 (k % 4) of the
  //     16-lane group m = lane / 16, k = lane % 16, rr = 4 (m / 2) + k / 4
  //     = ((row base + 8 (k % 2) + 16 (c ^ swz)) ^ (64 d)) + 16 ks rows (+ 8 rows),
  //     c = 2 (m % 2) + (k % 4) / 2.
  //   fp8: K step ss: row kb * 32 + lrow, bytes 16 ss + 8 half (chunk ss ^ swz);
  //   Vᵀ step (ks, d): source lane s of 16-lane group m addresses key 16 ks + kk,
  //   kk = 4 (m / 2) + {0, 1, 2, 3, 8, 9, 10, 11}[s / 2], the 8 bytes at dim
  //   32 d + 16 (m % 2) + 8 (s % 2): chunk (2 d + m % 2) ^ swz(kk), so lane j of the group
  //   receives dim 32 d + 16 (m % 2) + j of those eight keys, in P's key order.
  const int tr_k = lane & 15;
  const int tr_m = lane >> 4;
  uint32_t k_lane, v_lane;
  if constexpr (kFp8) {
    const int kb8 = tr_k >> 1;
    const int kk = 4 * (tr_m >> 1) + (kb8 & 3) + 8 * (kb8 >> 2);
    k_lane = lrow * RB + 16 * SW::k(lrow) + 8 * half;
    v_lane = kk * RB + 16 * ((tr_m & 1) ^ SW::v(kk)) + 8 * (tr_k & 1);
  } else {
    const int rr = (tr_m >> 1) * 4 + (tr_k >> 2);
    k_lane = lrow * RB + 16 * (half ^ SW::k(lrow));
    v_lane = rr * RB + 8 * (tr_k & 1) + 16 * ((2 * (tr_m & 1) + ((tr_k & 3) >> 1)) ^ SW::v(rr));
  }

  using Stage0 = std::integral_constant<int, 0>;
  using Stage1 = std::integral_constant<int, 1>;
  int32_t pg_next = page_of_tile(kt_begin);
  issue(tile_rsrc(kpool, kt_begin, pg_next), tile_rsrc(vpool, kt_begin, pg_next), Stage0{}, 0, kTileLoads);
  pg_next = page_of_tile(kt_begin + 1);
  auto tile = [&](auto stage, int kt) {
    constexpr int ST = decltype(stage)::value;
    using Next = std::integral_constant<int, 1 - ST>;
    // vmcnt(0): this wave's share of tile kt (and the next page id) has arrived
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();                 // all of tile kt is in LDS; the other stage is no longer read
    // At head_dim 256 (one wave per SIMD) the next tile's loads are spread over the MFMA
    // steps of phases A and B: issued all at once here, the four waves' loads queued at the
    // texture unit together and held every wave for about a quarter of the tile.  With two
    // waves per SIMD the other wave covers that, and one batch here measured faster.  Past
    // the last tile every page slot starts past the range, so the resources are empty and
    // the loads only write zeros into the stage that nothing reads any more.
    const __amdgpu_buffer_rsrc_t nk = tile_rsrc(kpool, kt + 1, pg_next), nv = tile_rsrc(vpool, kt + 1, pg_next);
    pg_next = page_of_tile(kt + 2);
    const int key0 = kt * kTileKeys;
    const bool masked = key0 > wave_last || key0 + kTileKeys <= wave_lo;   // for every row of this wave
    if (!kSpreadLoads || masked) issue(nk, nv, Next{}, 0, kTileLoads);
    if (masked) return;
    // loads of MFMA step u (0 <= u < 2 NS over phases A and B)
    auto issue_step = [&](int u) {
      if constexpr (kSpreadLoads)
        issue(nk, nv, Next{}, u * kTileLoads / (2 * NS), (u + 1) * kTileLoads / (2 * NS));
    };

    const lds_char* kbase = (const lds_char*)(lds_void*)(ST ? sB_K1 : sB_K0);
    const lds_char* vbase = (const lds_char*)(lds_void*)(ST ? sA_V1 : sA_V0);
    auto kread = [&](int kb, int ss) -> uint4 {
      if constexpr (kFp8) {
        const uint32_t addr = (k_lane ^ (uint32_t)(16 * ss)) + kb * 32 * RB;
        const u32x2 w = *reinterpret_cast<const lds_u32x2*>(kbase + addr);
        return widen_fp8x8(w.x, w.y);
      } else {
        const uint32_t addr = (k_lane ^ (uint32_t)(32 * ss)) + kb * 32 * RB;
        return __builtin_bit_cast(uint4, *reinterpret_cast<const lds_u32x4*>(kbase + addr));
      }
    };
    auto vread = [&](int t, uint4& dst) {     // step t = ks * ND + d
      const int ks = t / ND, d = t % ND;
      if constexpr (kFp8) {
        const uint32_t a1 = (v_lane ^ (uint32_t)(32 * d)) + ks * 16 * RB;
        const i32x2 w = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(vbase + a1));
        dst = widen_fp8x8((uint32_t)w.x, (uint32_t)w.y);
      } else {
        const uint32_t a1 = (v_lane ^ (uint32_t)(64 * d)) + ks * 16 * RB;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbase + a1));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbase + a1 + 8 * RB));
        const uint2 lo2 = __builtin_bit_cast(uint2, lo), hi2 = __builtin_bit_cast(uint2, hi);
        dst = make_uint4(lo2.x, lo2.y, hi2.x, hi2.y);
      }
    };

    // The tile's two 32-key blocks are pipelined so that each block's softmax (vector ALU)
    // overlaps matrix-core work of the other: S of block 0; S of block 1 beside the softmax
    // of block 0; P V of block 0 beside the softmax of block 1; P V of block 1.  The running
    // reference is updated per 32-key block (blocks sit at absolute multiples of 32 keys).
    // Each phase is one scheduling region (no branch inside), so the compiler interleaves the
    // vector work between the MFMAs; phases end at the wave-uniform mask and O-rescale
    // branches, the latter rare thanks to the lazy reference.
    // s[kb] takes both the K Q_hi and the K Q_lo products of block kb, one accumulation chain
    // (back-to-back MFMAs into the same registers issue at full rate; two alternating chains
    // measured slower)
    f32x16 s[2];
#pragma unroll
    for (int r = 0; r < 16; ++r) s[0][r] = s[1][r] = 0.0f;

    // causal / window mask of block kb, only on tiles that cross the causal diagonal or a
    // window's lower edge (a wave-uniform branch, kept out of the pipelined regions)
    const bool need_mask = key0 + kTileKeys - 1 > wave_first || key0 < mask_lo;
    auto mask_block = [&](int kb) {
      if (need_mask) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + kb * 32 + half * 4 + (r >> 2) * 8 + (r & 3);
          s[kb][r] = (key <= row_n && key >= row_lo) ? s[kb][r] : -INFINITY;
        }
      }
    };
    // softmax of block kb after its mask: the block's row max of the raw scores (the scale,
    // > 0, is folded into one FMA), then the lazy reference: a row's reference m (log2 units)
    // is raised only when the block max exceeds it by more than kRescale, so p = exp2(s *
    // scale - m) stays <= 2^kRescale and most blocks leave O alone; p is rounded to bf16 into
    // the P^T fragments pf[2 kb], pf[2 kb + 1] (this lane's keys q0 + 0..3 and q0 + 8..11,
    // q0 = 16 ks + 4 (lane / 32), in the accumulator's order); st.alpha is the O scale factor,
    // exactly 1 for a row whose reference stayed.
    // The work is cut into kSoftPieces pieces so that each sits beside one matrix step of the
    // other block, in a scheduling region of its own: left to itself the scheduler moved the
    // whole softmax behind the MFMAs it was meant to overlap.  Pieces 0-3: the max over four
    // scores each; 4: the max of both halves of the row, the reference and the factor; 5-12:
    // two exponentials each and their running sum (in key order); 13: the sum of both halves
    // and the running sum of the row; 14-15: the bf16 packing of eight values each.
    // Branch-free: exp2(-inf - finite) = 0 for a first raise, and the value of an unraised
    // lane (possibly NaN) is discarded by the select.
    uint4 pf[4];
    struct SoftState {
      float mx, alpha, m_ref, psum;
      bool raised;
    };
    auto soft_piece = [&](int kb, int j, SoftState& st) {
      if (j < 4) {
        if (j == 0) st.mx = -INFINITY;
#pragma unroll
        for (int r = 4 * j; r < 4 * j + 4; ++r) st.mx = fmaxf(st.mx, s[kb][r]);
      } else if (j == 4) {
        const float2 mh = halves32(st.mx);
        const float mx2 = fmaxf(mh.x, mh.y) * a.scale_log2;
        st.raised = mx2 > m_run + kRescale;
        st.alpha = st.raised ? __builtin_amdgcn_exp2f(m_run - mx2) : 1.0f;
        m_run = st.raised ? mx2 : m_run;
        // a row that has not seen a key yet (a windowed row whose window starts past this
        // block) has m = -inf and only -inf scores: its reference 0 gives p = 0, not NaN
        st.m_ref = (m_run == -INFINITY) ? 0.0f : m_run;
        st.psum = 0.0f;
      } else if (j < 13) {
#pragma unroll
        for (int r = 2 * (j - 5); r < 2 * (j - 5) + 2; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[kb][r], a.scale_log2, -st.m_ref));
          s[kb][r] = p;
          st.psum += p;
        }
      } else if (j == 13) {
        const float2 ph = halves32(st.psum);
        l_run = l_run * st.alpha + (ph.x + ph.y);
      } else {
        const int hs = j - 14;
        uint4& f = pf[2 * kb + hs];
        f.x = pack_bf16_rne(s[kb][8 * hs + 0], s[kb][8 * hs + 1]);
        f.y = pack_bf16_rne(s[kb][8 * hs + 2], s[kb][8 * hs + 3]);
        f.z = pack_bf16_rne(s[kb][8 * hs + 4], s[kb][8 * hs + 5]);
        f.w = pack_bf16_rne(s[kb][8 * hs + 6], s[kb][8 * hs + 7]);
      }
    };
    auto rescale_o = [&](bool raised, float alpha) {
      if (__builtin_amdgcn_ballot_w64(raised) != 0) {
#pragma unroll
        for (int d = 0; d < ND; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[d][r] *= alpha;
      }
    };

    // K fragments of both 32-key blocks form one stream (f = block * NS + k-step) read LK
    // fragments ahead of their MFMAs; Vᵀ fragments one stream (t = 16-key step * ND + d)
    // read LV ahead, the first LV of them issued with block 1's S so that phase C starts
    // on fragments that have long arrived.  At head_dim 256 one wave per SIMD leaves nothing
    // else to cover an LDS read, so the lookahead is deeper there.
    constexpr int LK = NS >= 16 ? kLookK256 : 2;
    constexpr int RK = LK + 1;
    constexpr int NT = 4 * ND;
    constexpr int LV = NS >= 16 ? kLookV256 : 3;
    constexpr int RV = LV + 1;
    uint4 kf[RK], vf[RV];
    auto kfetch = [&](int f) {
      if (f < 2 * NS) kf[f % RK] = kread(f / NS, f % NS);
    };
    auto vfetch = [&](int t) {
      if (t < NT) vread(t, vf[t % RV]);
    };
#pragma unroll
    for (int f = 0; f < LK; ++f) kfetch(f);

    // phase A: S of block 0
#pragma unroll
    for (int ss = 0; ss < NS; ++ss) {
      kfetch(ss + LK);
      issue_step(ss);
      __builtin_amdgcn_sched_barrier(0);
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[ss % RK]), as_bf16x8(qf[ss]), s[0], 0, 0, 0);
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[ss % RK]), as_bf16x8(ql[ss]), s[0], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    mask_block(0);

    // phase B: S of block 1 beside the softmax of block 0; the K stream's last LK fragments
    // are read in its first steps, the first LV Vᵀ fragments in its last
    constexpr int kSoftPieces = 16;
    static_assert(LV <= NS && kSoftPieces % NS == 0 && kSoftPieces % (2 * ND) == 0, "softmax pieces per step");
    SoftState st0, st1;
#pragma unroll
    for (int ss = 0; ss < NS; ++ss) {
      const int f = NS + ss;
      kfetch(f + LK);
      issue_step(NS + ss);
      if (ss >= NS - LV) vfetch(ss - (NS - LV));
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[f % RK]), as_bf16x8(qf[ss]), s[1], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[f % RK]), as_bf16x8(ql[ss]), s[1], 0, 0, 0);
#pragma unroll
      for (int j = ss * kSoftPieces / NS; j < (ss + 1) * kSoftPieces / NS; ++j) soft_piece(0, j, st0);
      __builtin_amdgcn_sched_barrier(0);
    }
    rescale_o(st0.raised, st0.alpha);
    mask_block(1);

    // phases C and D: O^T += V^T P^T over the four 16-key steps (block 0: ks 0, 1; block 1:
    // ks 2, 3); the softmax of block 1 beside phase C
#pragma unroll
    for (int t = 0; t < 2 * ND; ++t) {
      vfetch(t + LV);
      const int d = t % ND;
      o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vf[t % RV]), as_bf16x8(pf[t / ND]), o[d], 0, 0, 0);
#pragma unroll
      for (int j = t * kSoftPieces / (2 * ND); j < (t + 1) * kSoftPieces / (2 * ND); ++j) soft_piece(1, j, st1);
      __builtin_amdgcn_sched_barrier(0);
    }
    rescale_o(st1.raised, st1.alpha);
#pragma unroll
    for (int t = 2 * ND; t < NT; ++t) {
      vfetch(t + LV);
      __builtin_amdgcn_sched_barrier(0);
      const int d = t % ND;
      o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vf[t % RV]), as_bf16x8(pf[t / ND]), o[d], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  for (int kt = kt_begin; kt < n_tiles; kt += 2) {
    tile(Stage0{}, kt);
    if (kt + 1 < n_tiles) tile(Stage1{}, kt + 1);
  }

  // ---- shared split: the partial (reference, sum, unnormalised O) of this lane's row in the
  // decode's layout, for the combine kernel
  // (or, for the per-sequence part of a suffix prefill over shared pages, slot part_slot)
  if (kShared || (a.part_acc != nullptr && layer_window(a, l) == 0)) {
    if (row_ok) {
      const int slot = kShared ? split : a.part_slot;
      const int64_t pidx = ((((int64_t)l * a.batch + b) * a.chunk + row) * a.Hq + h) * a.n_split_max + slot;
      float* op = a.part_acc + pidx * D;
#pragma unroll
      for (int d = 0; d < ND; ++d)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
          *reinterpret_cast<float4*>(op + d * 32 + r4 * 8 + half * 4) =
              make_float4(o[d][r4 * 4 + 0], o[d][r4 * 4 + 1], o[d][r4 * 4 + 2], o[d][r4 * 4 + 3]);
      if (half == 0) *reinterpret_cast<float2*>(a.part_ml + pidx * 2) = make_float2(m_run, l_run);
    }
    return;
  }
  // ---- normalise and store: lane owns row `row`, dims d*32 + (r/4)*8 + half*4 + r%4
  if (row_ok) {
    const float inv = 1.0f / l_run;
    float* op = a.out + ((((int64_t)l * a.batch + b) * a.chunk + row) * a.Hq + h) * D;
#pragma unroll
    for (int d = 0; d < ND; ++d)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        float4 v;
        v.x = o[d][r4 * 4 + 0] * inv;
        v.y = o[d][r4 * 4 + 1] * inv;
        v.z = o[d][r4 * 4 + 2] * inv;
        v.w = o[d][r4 * 4 + 3] * inv;
        *reinterpret_cast<float4*>(op + d * 32 + r4 * 8 + half * 4) = v;
      }
  }
}

}  // namespace

template <typename T, bool kShared>
hipError_t launch_prefill_t(const PrefillArgs& a, hipStream_t stream) {
  const int64_t n_wg = kShared ? (int64_t)a.n_layers * a.Hkv * a.n_shared_split * a.n_qt
                               : (int64_t)a.n_layers * a.batch * a.Hkv * a.n_qt;
  if (n_wg <= 0) return hipSuccess;
  switch (a.D) {
    case 64: prefill_mfma_kernel<T, 64, 8, kShared><<<dim3((unsigned)n_wg), 64 * 8, 0, stream>>>(a); break;
    case 128: prefill_mfma_kernel<T, 128, 8, kShared><<<dim3((unsigned)n_wg), 64 * 8, 0, stream>>>(a); break;
    case 256: prefill_mfma_kernel<T, 256, 4, kShared><<<dim3((unsigned)n_wg), 64 * 4, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Waves per workgroup: 8 where a wave's registers leave two waves per SIMD (head_dim <= 128),
// so one K/V tile in LDS serves 256 (row, head) pairs; 4 at head_dim 256 (O and the queries'
// hi and lo parts alone take 256 registers per lane).
int prefill_mfma_waves(int D) { return D <= 128 ? 8 : 4; }

hipError_t launch_prefill_mfma(const PrefillArgs& a, int dtype, hipStream_t stream) {
  if (dtype == kDtypeBf16) return launch_prefill_t<uint16_t, false>(a, stream);
  if (dtype == kDtypeFp8) return launch_prefill_t<uint8_t, false>(a, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_shared_splits(const PrefillArgs& a, int dtype, hipStream_t stream) {
  if (dtype == kDtypeBf16) return launch_prefill_t<uint16_t, true>(a, stream);
  if (dtype == kDtypeFp8) return launch_prefill_t<uint8_t, true>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace kvg
