// Grouped-query attention on the vector ALUs, split over keys ("split-K"), used for decode
// (one new row per sequence) and for fp32 caches' prefill rows.
//
// Work item = (layer, sequence, row, KV head g, split s).  A split is the fixed logical
// key range [512 s, 512 s + 512) of that row's visible keys [0, n]; the split plan is a
// function of the row's own length only.  One 256-thread workgroup per work item:
//   - teams of TL lanes (16, or fewer for narrow rows) each own every NT-th key of the
//     split (key k0 + team + NT i); lane tl of a team holds 16-byte chunks tl, tl + TL, ...
//     of the D-wide K and V rows, so a team reads whole rows with 16-byte loads, and each
//     team keeps the next key's rows in flight while it computes the current one.
//   - q for the `group` query heads that share KV head g sits in registers (fp32).
//   - per key: partial dot products, an xor butterfly inside the team (every lane
//     ends with identical bits because each step adds the same two values), then an
//     online-softmax update of the team's running (max m, sum l, weighted V acc) in fp32,
//     with exp2 of pre-scaled scores.
//   - the team states are merged with a fixed xor tree inside each wavefront and then
//     wave 0..3 in order through LDS, and written as the split's partial.
// A second kernel merges the partials of each row in ascending split order.  Nothing
// depends on physical page ids or on how many rows/sequences share the launch, which is
// what makes the graft path and the fresh path produce the same bytes.
#include "kvg_device.h"
#include "kvg_launch.h"

#include <math.h>

namespace kvg {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

struct Soft {
  float m, l;
};

// Merge factor exp2(m_part - m_new); a part that saw no key has m = -inf and weight 0.
__device__ __forceinline__ float merge_factor(float m_part, float m_new) {
  return (m_part == -INFINITY) ? 0.0f : exp2f(m_part - m_new);
}

template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void attn_partial_kernel(const AttnArgs a) {
  constexpr int CH = Elem<T>::kPerVec;          // elements per 16-byte chunk
  constexpr int NCH = D / CH;                   // chunks per row
  constexpr int TL = NCH < 16 ? NCH : 16;       // lanes per key ("team")
  constexpr int CPL = NCH / TL;                 // chunks per lane
  constexpr int EPL = CPL * CH;                 // elements per lane
  constexpr int NT = kThreads / TL;             // teams per workgroup
  static_assert(CPL >= 1 && (64 % TL) == 0, "unsupported head_dim");

  // decompose the flat work index: s fastest, then g, row, batch, layer
  int64_t w = blockIdx.x;
  const int s = (int)(w % a.n_split_max);  w /= a.n_split_max;
  const int g = (int)(w % a.Hkv);          w /= a.Hkv;
  const int r = (int)(w % a.rows);         w /= a.rows;
  const int b = (int)(w % a.batch);        w /= a.batch;
  const int l = (int)w;

  const int ctx = a.ctx_lens[b];
  if (ctx < 0 || ctx > a.max_ctx_len) return;
  const int n_keys = ctx + r + 1;                 // keys [0, ctx + r] are visible
  const int k0 = s * kSplit;
  if (k0 >= n_keys) return;
  const int k1 = min(k0 + kSplit, n_keys);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int tl = lane % TL;
  const int team = threadIdx.x / TL;

  const int64_t row_id = ((int64_t)l * a.batch + b) * a.rows + r;
  // queries of the group, this lane's chunks tl, tl + TL, ...
  float q[G][EPL];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float* qp = a.q + (row_id * a.Hq + (int64_t)g * G + h) * D;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = tl + TL * i;
#pragma unroll
      for (int e = 0; e < CH; e += 4) {
        const float4 f = *reinterpret_cast<const float4*>(qp + c * CH + e);
        q[h][i * CH + e] = f.x;
        q[h][i * CH + e + 1] = f.y;
        q[h][i * CH + e + 2] = f.z;
        q[h][i * CH + e + 3] = f.w;
      }
    }
  }

  float acc[G][EPL];
  Soft st[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    st[h].m = -INFINITY;
    st[h].l = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[h][e] = 0.0f;
  }

  const int64_t lbase = (int64_t)(a.layer0 + l) * a.layer_elems;
  const T* kpool = reinterpret_cast<const T*>(a.k_pool) + lbase;
  const T* vpool = reinterpret_cast<const T*>(a.v_pool) + lbase;
  const int32_t* bt = a.block_tables + (int64_t)b * a.max_pages;

  // one key's K and V chunks for this lane; `ok` false for a bad page (key skipped)
  struct Row {
    uint4 k[CPL], v[CPL];
    bool ok;
  };
  auto load_row = [&](int j, Row& rw) {
    const int32_t page = bt[j / kPage];
    rw.ok = page >= 0 && page < a.n_pages;
    const int64_t roff = (((int64_t)(rw.ok ? page : 0) * a.Hkv + g) * kPage + (j % kPage)) * D;
#pragma unroll
    for (int i = 0; i < CPL; ++i) rw.k[i] = *reinterpret_cast<const uint4*>(kpool + roff + (tl + TL * i) * CH);
#pragma unroll
    for (int i = 0; i < CPL; ++i) rw.v[i] = *reinterpret_cast<const uint4*>(vpool + roff + (tl + TL * i) * CH);
  };
  auto consume = [&](const Row& rw) {
    if (!rw.ok) return;                               // uniform within a team
    float sc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) sc[h] = 0.0f;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
#pragma unroll
      for (int e = 0; e < CH; ++e) {
        const float kf = Elem<T>::get(rw.k[i], e);
#pragma unroll
        for (int h = 0; h < G; ++h) sc[h] = fmaf(q[h][i * CH + e], kf, sc[h]);
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int m = 1; m < TL; m <<= 1) sc[h] += __shfl_xor(sc[h], m);
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float s2 = sc[h] * a.scale_log2;
      const float m_new = fmaxf(st[h].m, s2);
      const float alpha = merge_factor(st[h].m, m_new);
      const float p = exp2f(s2 - m_new);
      st[h].l = fmaf(st[h].l, alpha, p);
      st[h].m = m_new;
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
#pragma unroll
        for (int e = 0; e < CH; ++e) {
          const float vf = Elem<T>::get(rw.v[i], e);
          acc[h][i * CH + e] = fmaf(acc[h][i * CH + e], alpha, p * vf);
        }
      }
    }
  };

  // keys k0 + team, k0 + team + NT, ...: two rows in flight per team
  int j = k0 + team;
  Row ra, rb;
  if (j < k1) load_row(j, ra);
  while (j < k1) {
    const int jn = j + NT;
    if (jn < k1) load_row(jn, rb);
    consume(ra);
    if (jn >= k1) break;
    const int jn2 = jn + NT;
    if (jn2 < k1) load_row(jn2, ra);
    consume(rb);
    j = jn2;
  }

  // merge the teams of this wavefront (lanes with equal tl hold equal chunks)
#pragma unroll
  for (int mask = TL; mask < 64; mask <<= 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float m_o = __shfl_xor(st[h].m, mask);
      const float l_o = __shfl_xor(st[h].l, mask);
      const float m_new = fmaxf(st[h].m, m_o);
      const float f_me = merge_factor(st[h].m, m_new);
      const float f_o = merge_factor(m_o, m_new);
      st[h].l = st[h].l * f_me + l_o * f_o;
      st[h].m = m_new;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float a_o = __shfl_xor(acc[h][e], mask);
        acc[h][e] = acc[h][e] * f_me + a_o * f_o;
      }
    }
  }

  // merge waves 0..3 in order through LDS
  __shared__ float s_acc[4][G][D];
  __shared__ float s_ml[4][G][2];
  if (lane < TL) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
#pragma unroll
        for (int e = 0; e < CH; ++e) s_acc[wave][h][(tl + TL * i) * CH + e] = acc[h][i * CH + e];
      }
      if (lane == 0) {
        s_ml[wave][h][0] = st[h].m;
        s_ml[wave][h][1] = st[h].l;
      }
    }
  }
  __syncthreads();

  const int64_t part_base = (row_id * a.Hq + (int64_t)g * G) * a.n_split_max + s;  // head 0 of group
  for (int t = threadIdx.x; t < G * D; t += kThreads) {
    const int h = t / D;
    const int d = t - h * D;
    float m = s_ml[0][h][0], lsum = s_ml[0][h][1], o = s_acc[0][h][d];
#pragma unroll
    for (int wv = 1; wv < 4; ++wv) {
      const float m_o = s_ml[wv][h][0];
      const float m_new = fmaxf(m, m_o);
      const float f_me = merge_factor(m, m_new);
      const float f_o = merge_factor(m_o, m_new);
      lsum = lsum * f_me + s_ml[wv][h][1] * f_o;
      o = o * f_me + s_acc[wv][h][d] * f_o;
      m = m_new;
    }
    const int64_t pidx = part_base + (int64_t)h * a.n_split_max;
    a.part_acc[pidx * D + d] = o;
    if (d == 0) {
      a.part_ml[pidx * 2] = m;
      a.part_ml[pidx * 2 + 1] = lsum;
    }
  }
}

// Combine a row's split partials in ascending split order and normalise.
__global__ __launch_bounds__(kThreads) void attn_merge_kernel(const AttnArgs a) {
  int64_t w = blockIdx.x;                       // (layer, batch, row, q head)
  const int h = (int)(w % a.Hq);   w /= a.Hq;
  const int r = (int)(w % a.rows); w /= a.rows;
  const int b = (int)(w % a.batch);
  const int64_t row_head = blockIdx.x;
  float* out = a.out + row_head * a.D;
  const int ctx = a.ctx_lens[b];
  if (ctx < 0 || ctx > a.max_ctx_len) {
    for (int d = threadIdx.x; d < a.D; d += kThreads) out[d] = __int_as_float(0x7FC00000);
    return;
  }
  const int n_keys = ctx + r + 1;
  const int n_split = (n_keys + kSplit - 1) / kSplit;
  const float* ml = a.part_ml + row_head * a.n_split_max * 2;
  const float* acc = a.part_acc + row_head * a.n_split_max * a.D;
  float m = -INFINITY;
  for (int s = 0; s < n_split; ++s) m = fmaxf(m, ml[2 * s]);
  for (int d = threadIdx.x; d < a.D; d += kThreads) {
    float lsum = 0.0f, o = 0.0f;
    for (int s = 0; s < n_split; ++s) {
      const float f = merge_factor(ml[2 * s], m);
      lsum = fmaf(ml[2 * s + 1], f, lsum);
      o = fmaf(acc[(int64_t)s * a.D + d], f, o);
    }
    out[d] = o / lsum;
  }
}

template <typename T, int D>
hipError_t launch_partial_g(const AttnArgs& a, hipStream_t stream) {
  const int64_t n_blocks = (int64_t)a.n_layers * a.batch * a.rows * a.Hkv * a.n_split_max;
  switch (a.group) {
    case 1: attn_partial_kernel<T, D, 1><<<dim3((unsigned)n_blocks), kThreads, 0, stream>>>(a); break;
    case 2: attn_partial_kernel<T, D, 2><<<dim3((unsigned)n_blocks), kThreads, 0, stream>>>(a); break;
    case 4: attn_partial_kernel<T, D, 4><<<dim3((unsigned)n_blocks), kThreads, 0, stream>>>(a); break;
    case 8: attn_partial_kernel<T, D, 8><<<dim3((unsigned)n_blocks), kThreads, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_partial_d(const AttnArgs& a, hipStream_t stream) {
  switch (a.D) {
    case 64: return launch_partial_g<T, 64>(a, stream);
    case 128: return launch_partial_g<T, 128>(a, stream);
    case 256: return launch_partial_g<T, 256>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attn_valu(const AttnArgs& a, int bf16, hipStream_t stream) {
  hipError_t e = bf16 ? launch_partial_d<uint16_t>(a, stream) : launch_partial_d<float>(a, stream);
  if (e != hipSuccess) return e;
  const int64_t n_rows = (int64_t)a.n_layers * a.batch * a.rows * a.Hq;
  attn_merge_kernel<<<dim3((unsigned)n_rows), kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace kvg
