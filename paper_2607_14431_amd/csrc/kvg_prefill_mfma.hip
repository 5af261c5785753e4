// Chunked-prefill attention on bf16 MFMA (gfx950 v_mfma_f32_32x32x16_bf16) over a paged
// cache: the suffix rows attend causally to the cached (e.g. grafted) prefix and to the
// chunk itself.
//
// Workgroup = (layer, sequence, KV head g, q-tile).  A q-tile holds BM = 128 / group query
// rows for each of the `group` query heads that share KV head g, so one K/V tile in LDS
// serves 128 (row, head) pairs; wave w owns 32 consecutive rows of one head.
//
// Per 64-key tile (tiles start at absolute multiples of 64 of the logical key index, so a
// row's arithmetic does not depend on how the sequence was chunked):
//   S^T = K Q^T   A = K rows from LDS (row-major, rows padded by 16 B), B = the wave's
//                 queries held in registers; C = 32 keys x 32 rows, so each lane owns one
//                 query row (lane % 32) and 16 of its keys, the other half in lane ^ 32.
//   softmax       causal mask (key <= row), running reference / sum per row in fp32 with
//                 exp2 (scale folded into one FMA); both halves of a row exchange their tile
//                 max and sum; the reference moves only when a tile max exceeds it by 2^8,
//                 so most tiles skip the O rescale.
//   O^T += V^T P^T  A = V^T from LDS (transposed while staging: 8x8 bf16 blocks per lane,
//                 rows padded to 136 B), B = P rounded to bf16 straight from the S^T
//                 registers (the key order inside each 16-key step is the accumulator's
//                 own order, used identically for both operands); C = O^T, one row per lane
//                 so the rescale by exp2(m_old - m_new) is a per-lane multiply.
// The next tile's K/V are loaded into registers while the current tile is computed.
// Keys past the workgroup's last row are zero-filled in LDS so no poison reaches P V.
#include "kvg_device.h"
#include "kvg_launch.h"

#include <math.h>

namespace kvg {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kTileKeys = 64;
constexpr float kRescale = 8.0f;  // lazy-rescale threshold of a row's reference (log2 units)
constexpr int kVtRowU2 = 17;     // V^T tile row stride in uint2 (136 B: 128 + 8 pad)

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// two fp32 -> packed bf16, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16_rne(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

template <int D>
struct TileRegs {
  static constexpr int kK = (kTileKeys * D / 8) / kThreads;     // 16-byte K chunks per thread
  static constexpr int kVBlocks = (8 * (D / 8) + kThreads - 1) / kThreads;  // 8x8 V blocks per thread
  uint4 k[kK];
  uint4 v[kVBlocks][8];
};

template <int D>
__global__ __launch_bounds__(kThreads) void prefill_mfma_kernel(const PrefillArgs a) {
  constexpr int NCH = D / 8;           // 16-byte chunks per row
  constexpr int NS = D / 16;           // MFMA k-steps over head_dim
  constexpr int ND = D / 32;           // 32-wide blocks of head_dim
  constexpr int kKRowU4 = NCH + 1;     // K tile row stride in uint4: one 16-byte pad per row
  __shared__ uint4 sK[kTileKeys * kKRowU4];
  __shared__ uint2 sVt[D * kVtRowU2];

  // ---- workgroup coordinates: XCD-aware order, heavy (late) q-tiles first
  const int nwg = gridDim.x;
  int id = blockIdx.x;
  const int per_xcd = nwg / 8;
  if (id < per_xcd * 8) id = (id % 8) * per_xcd + id / 8;
  int qt = id % a.n_qt;
  int rest = id / a.n_qt;
  const int g = rest % a.Hkv;
  rest /= a.Hkv;
  const int b = rest % a.batch;
  const int l = rest / a.batch;
  qt = a.n_qt - 1 - qt;

  const int ctx = a.ctx_lens[b];
  if (ctx < 0 || ctx > a.max_ctx_len) return;
  const int G = a.group;
  const int BM = 128 / G;
  const int i0 = qt * BM;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int lrow = lane & 31;
  const int half = lane >> 5;
  const int h_local = (wave * 32) / BM;
  const int r0 = (wave * 32) % BM;
  const int h = g * G + h_local;
  const int row = i0 + r0 + lrow;                       // chunk row of this lane
  const int row_n = ctx + row;                          // its logical index: keys [0, row_n]
  const int wave_last = ctx + min(i0 + r0 + 31, a.chunk - 1);   // last key any row of this wave sees
  const int n_hi = ctx + min(i0 + BM, a.chunk);         // keys [0, n_hi) needed by the workgroup
  const int n_tiles = (n_hi + kTileKeys - 1) / kTileKeys;

  const int64_t lbase = (int64_t)(a.layer0 + l) * a.layer_elems;
  const uint16_t* kpool = reinterpret_cast<const uint16_t*>(a.k_pool) + lbase;
  const uint16_t* vpool = reinterpret_cast<const uint16_t*>(a.v_pool) + lbase;
  const int32_t* bt = a.block_tables + (int64_t)b * a.max_pages;

  // ---- queries of this lane's row (B operand of S^T = K Q^T), zeros past the chunk
  uint4 qf[NS];
  {
    const bool ok = row < a.chunk;
    const uint16_t* qp = a.q + ((((int64_t)l * a.batch + b) * a.chunk + (ok ? row : 0)) * a.Hq + h) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      qf[s] = ok ? *reinterpret_cast<const uint4*>(qp + (2 * s + half) * 8) : make_uint4(0, 0, 0, 0);
  }

  f32x16 o[ND];
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[d][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  // ---- tile staging
  auto row_ptr = [&](const uint16_t* pool, int key, bool& ok) -> const uint16_t* {
    ok = key < n_hi;
    if (!ok) return pool;
    const int32_t page = bt[key / kPage];
    ok = page >= 0 && page < a.n_pages;
    return pool + (((int64_t)(ok ? page : 0) * a.Hkv + g) * kPage + (key % kPage)) * D;
  };
  TileRegs<D> tr;
  auto load_tile = [&](int kt) {
    const int key0 = kt * kTileKeys;
#pragma unroll
    for (int j = 0; j < TileRegs<D>::kK; ++j) {
      const int cid = tid + j * kThreads;
      const int key = cid / NCH, c = cid % NCH;
      bool ok;
      const uint16_t* p = row_ptr(kpool, key0 + key, ok);
      tr.k[j] = ok ? *reinterpret_cast<const uint4*>(p + c * 8) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int vb = 0; vb < TileRegs<D>::kVBlocks; ++vb) {
      const int blk = tid + vb * kThreads;          // (key group kg, d chunk c)
      if (blk < 8 * NCH) {
        const int kg = blk / NCH, c = blk % NCH;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          bool ok;
          const uint16_t* p = row_ptr(vpool, key0 + kg * 8 + j, ok);
          tr.v[vb][j] = ok ? *reinterpret_cast<const uint4*>(p + c * 8) : make_uint4(0, 0, 0, 0);
        }
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int j = 0; j < TileRegs<D>::kK; ++j) {
      const int cid = tid + j * kThreads;
      sK[(cid / NCH) * kKRowU4 + (cid % NCH)] = tr.k[j];
    }
#pragma unroll
    for (int vb = 0; vb < TileRegs<D>::kVBlocks; ++vb) {
      const int blk = tid + vb * kThreads;
      if (blk < 8 * NCH) {
        const int kg = blk / NCH, c = blk % NCH;
        // transpose 8 keys x 8 dims: out[e] = the 8 keys of dimension 8c + e
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint32_t w[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t x0 = (&tr.v[vb][2 * j].x)[e >> 1];
            const uint32_t x1 = (&tr.v[vb][2 * j + 1].x)[e >> 1];
            w[j] = (e & 1) ? ((x0 >> 16) | (x1 & 0xFFFF0000u)) : ((x0 & 0xFFFFu) | (x1 << 16));
          }
          uint2* dst = &sVt[(c * 8 + e) * kVtRowU2 + kg * 2];
          dst[0] = make_uint2(w[0], w[1]);
          dst[1] = make_uint2(w[2], w[3]);
        }
      }
    }
  };

  load_tile(0);
  for (int kt = 0; kt < n_tiles; ++kt) {
    __syncthreads();                 // previous tile's LDS reads are complete
    store_tile();
    __syncthreads();
    if (kt + 1 < n_tiles) load_tile(kt + 1);
    const int key0 = kt * kTileKeys;
    if (key0 > wave_last) continue;  // tile fully masked for every row of this wave

    // S^T = K Q^T : two 32-key blocks
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.0f;
#pragma unroll
      for (int st = 0; st < NS; ++st) {
        const uint4 kf = sK[(kb * 32 + lrow) * kKRowU4 + 2 * st + half];
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf), as_bf16x8(qf[st]), s[kb], 0, 0, 0);
      }
    }

    // causal mask and the tile's row max (raw scores; the scale is folded into one FMA
    // below since scale > 0 commutes with max)
    const bool need_mask = key0 + kTileKeys - 1 > ctx + i0 + r0;   // some key may exceed some row
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = s[kb][r];
        if (need_mask) {
          const int key = key0 + kb * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
          v = (key <= row_n) ? v : -INFINITY;
        }
        s[kb][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    // lazy reference: the row's reference (log2 units) is raised only when the tile max
    // exceeds it by more than kRescale, so p = exp2(s * scale - m) stays <= 2^kRescale and
    // most tiles skip the O rescale; rows that keep their reference multiply by exactly 1
    const float mx2 = mx * a.scale_log2;
    const bool raise = mx2 > m_run + kRescale;
    float alpha = 1.0f;
    if (raise) {
      alpha = (m_run == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m_run - mx2);
      m_run = mx2;
    }
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
      l_run *= alpha;
#pragma unroll
      for (int d = 0; d < ND; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[d][r] *= alpha;
    }
    float psum = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[kb][r], a.scale_log2, -m_run));
        s[kb][r] = p;
        psum += p;
      }
    psum += __shfl_xor(psum, 32);
    l_run += psum;

    // O^T += V^T P^T : four 16-key steps
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int kb = ks >> 1, hs = ks & 1;
      uint4 pf;
      pf.x = pack_bf16_rne(s[kb][8 * hs + 0], s[kb][8 * hs + 1]);
      pf.y = pack_bf16_rne(s[kb][8 * hs + 2], s[kb][8 * hs + 3]);
      pf.z = pack_bf16_rne(s[kb][8 * hs + 4], s[kb][8 * hs + 5]);
      pf.w = pack_bf16_rne(s[kb][8 * hs + 6], s[kb][8 * hs + 7]);
      const int q4 = kb * 8 + hs * 4 + half;        // first 4-key group of this lane's keys
#pragma unroll
      for (int d = 0; d < ND; ++d) {
        const uint2* vr = &sVt[(d * 32 + lrow) * kVtRowU2];
        const uint2 v0 = vr[q4];
        const uint2 v1 = vr[q4 + 2];
        const uint4 vf = make_uint4(v0.x, v0.y, v1.x, v1.y);
        o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vf), as_bf16x8(pf), o[d], 0, 0, 0);
      }
    }
  }

  // ---- normalise and store: lane owns row `row`, dims d*32 + (r/4)*8 + half*4 + r%4
  if (row < a.chunk) {
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

hipError_t launch_prefill_mfma(const PrefillArgs& a, hipStream_t stream) {
  const int64_t n_wg = (int64_t)a.n_layers * a.batch * a.Hkv * a.n_qt;
  switch (a.D) {
    case 64: prefill_mfma_kernel<64><<<dim3((unsigned)n_wg), kThreads, 0, stream>>>(a); break;
    case 128: prefill_mfma_kernel<128><<<dim3((unsigned)n_wg), kThreads, 0, stream>>>(a); break;
    case 256: prefill_mfma_kernel<256><<<dim3((unsigned)n_wg), kThreads, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kvg
