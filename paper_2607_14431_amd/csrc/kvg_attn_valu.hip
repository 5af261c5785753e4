// Grouped-query attention on the vector ALUs, split over keys ("split-K"): the fused decode
// kernel (one new token per sequence) and the fp32 caches' prefill rows.
//
// Work item = (layer, sequence, row, KV head g, split s).  A split is the fixed logical
// key range [512 s, 512 s + 512) of the row's visible keys [0, n]; the split plan is a
// function of the row's own length only.  One 256-thread workgroup per work item:
//   - teams of TL lanes (16, or fewer for narrow rows) each own every NT-th key of the
//     split (key k0 + team + NT i); lane tl of a team holds 16-byte chunks tl, tl + TL, ...
//     of the D-wide K and V rows, so a team reads whole rows with 16-byte loads, and each
//     team keeps up to four keys' rows in flight while it computes.
//   - q for the `group` query heads that share KV head g sits in registers: for bf16 and
//     fp8 caches as packed bf16 hi and lo parts (each rotated value is hi + lo to 16
//     significant bits; a score is two v_dot2_f32_bf16 chains, hi and lo, with fp32
//     accumulation, added at the end), fp32 otherwise.  fp8 rows are widened to bf16 pairs when consumed (exact: every E4M3 value
//     is a bf16 value), so an fp8 cache reads half the bytes and computes like a bf16 one.
//   - per key: partial dot products, an xor butterfly inside the team (every lane ends
//     with identical bits because each step adds the same two values), then an online
//     softmax update of the team's running (reference m, sum l, weighted V acc) in fp32
//     with exp2 of pre-scaled scores; the reference m is raised only when a score exceeds
//     it by more than 2^8, so most keys cost one exp2 and one FMA per element.
//   - the team states are merged with a fixed xor tree inside each wavefront, then waves
//     0..3 in order through LDS.
// Splits are combined in ascending split order.  Nothing depends on physical page ids or
// on how many rows/sequences share the launch, which is what makes the graft path and the
// fresh path produce the same bytes.
#include "kvg_device.h"
#include "kvg_launch.h"

#include <math.h>

#include <algorithm>
#include <type_traits>

namespace kvg {

namespace {

constexpr int kThreads = 256;
constexpr float kRescale = 8.0f;     // lazy-rescale threshold of the running reference (log2 units)

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
// Cached K/V rows are read once per call: streaming (nontemporal) loads.  Measured on the
// 12B-class decode (1.83 GB per call over random pages): 326 -> 300 us per call.
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_stream(const void* p) {
  const u32x4v v = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
// c ? a : b per 32-bit component (a select of uint4 lvalues would select addresses and
// keep the operands in memory)
__device__ __forceinline__ uint4 sel4(bool c, const uint4& a, const uint4& b) {
  return make_uint4(c ? a.x : b.x, c ? a.y : b.y, c ? a.z : b.z, c ? a.w : b.w);
}
__device__ __forceinline__ void st16(void* p, const uint4& v) { *reinterpret_cast<uint4*>(p) = v; }

struct Soft {
  float m, l;
};

// Sum over the TL lanes of a team (TL = 4, 8 or 16 consecutive lanes) with DPP moves:
// partners lane ^ 1 and lane ^ 2 inside each quad, then the mirrored lane inside each half
// row and row.  After the quad steps all lanes of a quad hold the same bits, so the mirror
// steps pair the same two values an xor-4 / xor-8 butterfly would; every step adds the same
// two values in both partner lanes, so the whole team ends with identical bits.
template <int TL>
__device__ __forceinline__ float team_sum(float x) {
  static_assert(TL == 4 || TL == 8 || TL == 16, "team width");
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, true));
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x4E, 0xF, 0xF, true));
  if constexpr (TL >= 8)
    x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x141, 0xF, 0xF, true));
  if constexpr (TL >= 16)
    x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x140, 0xF, 0xF, true));
  return x;
}

// Page ids of a split's keys (at most kSplit / kPage + 1 pages, a window's split starting
// inside a page): lane i of every wave holds the page of logical page `first` + i, read
// once, so the key-row loads never wait on a block-table read.  The teams of one wave
// always read keys of the same logical page at a time, so the page of a key is taken with a
// lane read.
struct SplitPages {
  static_assert(kSplit / kPage + 1 <= 64, "a split's pages must fit a wave");
  int32_t pg;
  int base;
  // the block-table entries of the 64 pages from page `first` on, clamped to the table's
  // n_table entries (entries past the context are never used)
  __device__ __forceinline__ void init(const int32_t* bt, int first, int n_table, int lane) {
    base = first;
    pg = bt[min(base + lane, n_table - 1)];
  }
  __device__ __forceinline__ int32_t page_of(int j) const {
    const int i = __builtin_amdgcn_readfirstlane(j / kPage - base);
    return __builtin_amdgcn_readlane(pg, i);
  }
};

// Merge factor exp2(m_part - m_new); a part that saw no key has m = -inf and weight 0.
__device__ __forceinline__ float merge_factor(float m_part, float m_new) {
  return (m_part == -INFINITY) ? 0.0f : exp2f(m_part - m_new);
}

// Chunk of a cache row as bf16 pairs (32-bit words, element order): bf16 chunks are
// already that; an fp8 chunk (16 values) widens to 8 words, exactly.
template <typename T>
__device__ __forceinline__ void bf16_words(const uint4& c, uint32_t* w) {
  if constexpr (sizeof(T) == 1) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int x = (int)(&c.x)[j];
      w[2 * j] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, false));
      w[2 * j + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, true));
    }
  } else {
    w[0] = c.x;
    w[1] = c.y;
    w[2] = c.z;
    w[3] = c.w;
  }
}

template <typename T, int D, int G>
struct SplitWorker {
  static constexpr int CH = Elem<T>::kPerVec;     // elements per 16-byte chunk
  static constexpr int NCH = D / CH;              // chunks per row
  static constexpr int TL = NCH < 16 ? NCH : 16;  // lanes per key ("team")
  static constexpr int CPL = NCH / TL;            // chunks per lane
  static constexpr int EPL = CPL * CH;            // elements per lane
  static constexpr int NT = kThreads / TL;        // teams per workgroup
  static constexpr bool kBf16 = sizeof(T) <= 2;   // packed bf16 arithmetic (bf16 and fp8 caches)
  static constexpr int WPC = CH / 2;              // bf16 pairs per chunk (packed arithmetic)
  using QD = typename RawOf<T>::type;             // query dtype: bf16 for fp8 caches
  static constexpr int QC = CH / Elem<QD>::kPerVec;   // query chunks per cache chunk
  static constexpr int QW = kBf16 ? CPL * WPC : EPL;
  // key pairs in flight per team (the consumption order, and so the arithmetic, does not
  // depend on it; four pairs for fp8 rows measured no faster than two)
  static constexpr int kPairs = 2;
  static_assert(CPL >= 1 && (64 % TL) == 0 && TL >= 4, "unsupported head_dim");
  // a wave's teams never straddle a logical page: (64 / TL) teams per wave divide 16
  static_assert(kThreads / TL >= kPage, "teams per workgroup");
  using QT = typename std::conditional<kBf16, uint32_t, float>::type;

  struct Row {
    uint4 k[CPL], v[CPL];
    bool ok;
    bool lds;          // the new decode token: rows come from LDS when consumed
  };

  QT q[G][QW];
  uint32_t ql[kBf16 ? G : 1][kBf16 ? QW : 1];   // bf16 caches: the queries' lo parts
  float acc[G][EPL];
  Soft st[G];
  int tl, team, lane, wave;
  const uint4* lds_k = nullptr;   // the new token's K/V rows (16-byte chunks) in LDS
  const uint4* lds_v = nullptr;

  __device__ __forceinline__ void init() {
    lane = threadIdx.x & 63;
    wave = threadIdx.x >> 6;
    tl = lane % TL;
    team = threadIdx.x / TL;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      st[h].m = -INFINITY;
      st[h].l = 0.0f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[h][e] = 0.0f;
    }
  }

  // Query chunk j of this lane (16 bytes of QD): the lane's cache chunk j / QC, part
  // j % QC.  q_chunk(j) is its index among the row's D / kPerVec(QD) query chunks.
  __device__ __forceinline__ int q_chunk(int j) const { return (tl + TL * (j / QC)) * QC + j % QC; }
  // v: the chunk (bf16 hi parts for bf16 and fp8 caches), vl: the lo parts (bf16 only)
  __device__ __forceinline__ void set_q(int h, int j, const uint4& v, const uint4& vl) {
    if constexpr (kBf16) {
      q[h][j * 4 + 0] = v.x;
      q[h][j * 4 + 1] = v.y;
      q[h][j * 4 + 2] = v.z;
      q[h][j * 4 + 3] = v.w;
      ql[h][j * 4 + 0] = vl.x;
      ql[h][j * 4 + 1] = vl.y;
      ql[h][j * 4 + 2] = vl.z;
      ql[h][j * 4 + 3] = vl.w;
    } else {
      q[h][j * 4 + 0] = __uint_as_float(v.x);
      q[h][j * 4 + 1] = __uint_as_float(v.y);
      q[h][j * 4 + 2] = __uint_as_float(v.z);
      q[h][j * 4 + 3] = __uint_as_float(v.w);
    }
  }

  // Branches in the consume functions are uniform over the wavefront (ballots), so the
  // loads of later rows stay in flight across them.  A key that is not ok contributes
  // p = 0: its row is a real key's row (a key past the split loads key k1 - 1; the
  // decode's new token is taken from LDS), so 0 * V adds nothing.  Only a block-table
  // entry outside the pool (whose outputs are unspecified) can bring other bytes.
  __device__ __forceinline__ void fix_row(Row& rw) {
    if (__builtin_amdgcn_ballot_w64(rw.lds) != 0) {
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        const uint4 lk = lds_k[tl + TL * i], lv = lds_v[tl + TL * i];
        rw.k[i] = sel4(rw.lds, lk, rw.k[i]);
        rw.v[i] = sel4(rw.lds, lv, rw.v[i]);
      }
    }
  }

  // the key's scores for the G heads (log2 units), -inf for a key that is not ok
  __device__ __forceinline__ void scores(const Row& rw, float scale_log2, float (&s2)[G]) {
    float sc[G], sl[G];
#pragma unroll
    for (int h = 0; h < G; ++h) sc[h] = sl[h] = 0.0f;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      if constexpr (kBf16) {
        uint32_t kw[WPC];
        bf16_words<T>(rw.k[i], kw);
#pragma unroll
        for (int dw = 0; dw < WPC; ++dw)
#pragma unroll
          for (int h = 0; h < G; ++h) {
            sc[h] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, q[h][i * WPC + dw]),
                                                    __builtin_bit_cast(bf16x2, kw[dw]), sc[h], false);
            sl[h] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, ql[h][i * WPC + dw]),
                                                    __builtin_bit_cast(bf16x2, kw[dw]), sl[h], false);
          }
      } else {
#pragma unroll
        for (int e = 0; e < CH; ++e) {
          const float kf = Elem<T>::get(rw.k[i], e);
#pragma unroll
          for (int h = 0; h < G; ++h) sc[h] = fmaf(q[h][i * CH + e], kf, sc[h]);
        }
      }
    }
    if constexpr (kBf16) {
#pragma unroll
      for (int h = 0; h < G; ++h) sc[h] += sl[h];
    }
#pragma unroll
    for (int h = 0; h < G; ++h) s2[h] = rw.ok ? team_sum<TL>(sc[h]) * scale_log2 : -INFINITY;
  }

  // lazy rescale: the running reference only moves when a score exceeds it by more than
  // kRescale, so p = exp2(s2 - m) stays <= 2^kRescale; lanes that keep their reference
  // multiply by exactly 1
  __device__ __forceinline__ void raise_to(int h, float mx) {
    const bool raise = mx > st[h].m + kRescale;
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
      const float alpha = raise ? ((st[h].m == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(st[h].m - mx)) : 1.0f;
      st[h].m = raise ? mx : st[h].m;
      st[h].l *= alpha;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[h][e] *= alpha;
    }
  }

  // fp32 caches: one key, p and the weighted V in fp32
  __device__ __forceinline__ void consume(Row& rw, float scale_log2) {
    fix_row(rw);
    float s2[G];
    scores(rw, scale_log2, s2);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      raise_to(h, s2[h]);
      const float p = rw.ok ? __builtin_amdgcn_exp2f(s2[h] - st[h].m) : 0.0f;
      st[h].l += p;
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
#pragma unroll
        for (int e = 0; e < CH; ++e) acc[h][i * CH + e] = fmaf(p, Elem<T>::get(rw.v[i], e), acc[h][i * CH + e]);
      }
    }
  }

  // bf16 caches: two keys a, b.  Their weights are rounded to bf16 (as the MFMA prefill
  // rounds P) and the sum takes the rounded values, so the output stays a normalised
  // average; acc[e] += pa v_a[e] + pb v_b[e] is one v_dot2_f32_bf16 on (pa, pb) and the
  // pair (v_a[e], v_b[e]) assembled by one byte permute.
  __device__ __forceinline__ void consume_pair(Row& ra, Row& rb, float scale_log2) {
    fix_row(ra);
    fix_row(rb);
    float sa[G], sb[G];
    scores(ra, scale_log2, sa);
    scores(rb, scale_log2, sb);
    uint32_t va[CPL][WPC], vb[CPL][WPC];            // V rows as bf16 pairs, shared by the heads
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      bf16_words<T>(ra.v[i], va[i]);
      bf16_words<T>(rb.v[i], vb[i]);
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      raise_to(h, fmaxf(sa[h], sb[h]));
      const float pa = ra.ok ? __builtin_amdgcn_exp2f(sa[h] - st[h].m) : 0.0f;
      const float pb = rb.ok ? __builtin_amdgcn_exp2f(sb[h] - st[h].m) : 0.0f;
      const bf16x2 pp = __builtin_convertvector((f32x2){pa, pb}, bf16x2);
      st[h].l += (float)pp.x;
      st[h].l += (float)pp.y;
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
#pragma unroll
        for (int dw = 0; dw < WPC; ++dw) {
          // (v_a[2dw], v_b[2dw]) and (v_a[2dw+1], v_b[2dw+1]) as bf16 pairs
          const uint32_t lo = __builtin_amdgcn_perm(vb[i][dw], va[i][dw], 0x05040100u);
          const uint32_t hi = __builtin_amdgcn_perm(vb[i][dw], va[i][dw], 0x07060302u);
          float& a0 = acc[h][i * CH + 2 * dw];
          float& a1 = acc[h][i * CH + 2 * dw + 1];
          a0 = __builtin_amdgcn_fdot2_f32_bf16(pp, __builtin_bit_cast(bf16x2, lo), a0, false);
          a1 = __builtin_amdgcn_fdot2_f32_bf16(pp, __builtin_bit_cast(bf16x2, hi), a1, false);
        }
      }
    }
  }

  __device__ __forceinline__ void consume2(Row& ra, Row& rb, float scale_log2) {
    if constexpr (kBf16) {
      consume_pair(ra, rb, scale_log2);
    } else {
      consume(ra, scale_log2);
      consume(rb, scale_log2);
    }
  }

  // Keys k0 + team, k0 + team + NT, ... below k1, in stages of two keys with kPairs stages
  // (2 kPairs rows) in flight per team.  load(j, row) fills a row for a key j < k1.  Every
  // fetch is unconditional, so the loads stay in flight across the loop's back edge: a key
  // past k1 loads the row of key k1 - 1 (the same L2-resident row for every team) and is
  // marked not ok, which consume() turns into an exact no-op.  prologue() runs after the
  // first stages are in flight, so per-workgroup setup overlaps their latency; the queries
  // must be set by the time it returns.
  template <class Load, class Prologue>
  __device__ __forceinline__ void run(int k0, int k1, float scale_log2, Load load, Prologue prologue) {
    auto fetch = [&](int j, Row& rw) {
      const bool in = j < k1;
      load(in ? j : k1 - 1, rw);
      rw.ok = rw.ok && in;
    };
    const int n_it = (k1 - k0 + NT - 1) / NT;     // keys per team, rounded up
    constexpr int R = 2 * kPairs;                 // rows in flight per team
    Row rows[R];
    int j = k0 + team;
#pragma unroll
    for (int r = 0; r < R; ++r) fetch(j + r * NT, rows[r]);
    __builtin_amdgcn_sched_barrier(0);
    prologue();
    // Keys are consumed in order, a pair at a time; each pair's rows are refetched R keys
    // ahead as soon as they are consumed.  The scheduling barriers keep each stage's loads
    // where they are issued here (the scheduler would otherwise sink them to the end of the
    // body to shorten live ranges).
    for (int it = 0; it < n_it; it += R) {
#pragma unroll
      for (int p = 0; p < kPairs; ++p) {
        consume2(rows[2 * p], rows[2 * p + 1], scale_log2);
        __builtin_amdgcn_sched_barrier(0);
        fetch(j + (R + 2 * p) * NT, rows[2 * p]);
        fetch(j + (R + 2 * p + 1) * NT, rows[2 * p + 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
      j += R * NT;
    }
  }

  // Merge the teams of each wavefront (xor tree over lanes with equal tl) and leave each
  // wave's state in LDS: s_acc[wave][h][d], s_ml[wave][h] = (m, l).
  __device__ __forceinline__ void to_lds(float (*s_acc)[G][D], float (*s_ml)[G][2]) {
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
  }
};

// The split's state for (head h, element d): waves 0..3 merged in order.
template <int G, int D>
__device__ __forceinline__ void wave_merge(const float (*s_acc)[G][D], const float (*s_ml)[G][2], int h, int d,
                                           float& m, float& lsum, float& o) {
  m = s_ml[0][h][0];
  lsum = s_ml[0][h][1];
  o = s_acc[0][h][d];
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
}

// Final value of one output element from the splits' (m, l) pairs and weighted-V values
// (acc[s * acc_stride]), combined in ascending split order.
// Splits are taken U (eight unless the caller knows fewer) at a time with every load issued
// before its use: indices past the last split re-read the last one (a repeat changes no
// maximum) and are not added.  The sums run over the splits in ascending order whatever
// the unrolling, so every path that combines the same partials gives the same bytes.
template <int U = 8>
__device__ __forceinline__ float combine_splits(const float* ml, const float* acc, int64_t acc_stride, int n_split) {
  float m = -INFINITY;
  for (int s0 = 0; s0 < n_split; s0 += U) {
    float mv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) mv[u] = ml[2 * min(s0 + u, n_split - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u) m = fmaxf(m, mv[u]);
  }
  float lsum = 0.0f, o = 0.0f;
  for (int s0 = 0; s0 < n_split; s0 += U) {
    float2 pv[U];
    float av[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = min(s0 + u, n_split - 1);
      pv[u] = *reinterpret_cast<const float2*>(ml + 2 * s);
      av[u] = acc[s * acc_stride];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float f = merge_factor(pv[u].x, m);
      const bool in = s0 + u < n_split;
      lsum = in ? fmaf(pv[u].y, f, lsum) : lsum;
      o = in ? fmaf(av[u], f, o) : o;
    }
  }
  return o / lsum;
}

// ------------------------------------------------------------------------------------
// Multi-row calls (fp32 prefill): queries pre-rotated by the append kernel; each work item
// writes its split partial, combined by attn_merge_kernel.
template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void attn_partial_kernel(const AttnArgs a) {
  using W = SplitWorker<T, D, G>;
  int64_t w = blockIdx.x;
  const int s = (int)(w % a.n_split_max);  w /= a.n_split_max;
  const int g = (int)(w % a.Hkv);          w /= a.Hkv;
  const int r = (int)(w % a.rows);         w /= a.rows;
  const int b = (int)(w % a.batch);        w /= a.batch;
  const int l = (int)w;

  const int ctx = a.ctx_lens[b];
  if (ctx < 0 || ctx > a.max_ctx_len) return;
  const int n_keys = ctx + r + 1;                 // keys [0, ctx + r] are visible
  const int lo = window_start(layer_window(a, l), n_keys);
  if (s >= split_count(n_keys, lo)) return;
  const int k0 = lo + s * kSplit;                 // the split's keys [k0, k1)
  const int k1 = min(k0 + kSplit, n_keys);
  const int kb = k0 & ~(kPage - 1);               // teams start at the page holding k0

  W wk;
  wk.init();
  const int64_t row_id = ((int64_t)l * a.batch + b) * a.rows + r;
  constexpr int kQWordsPerRow = W::kBf16 ? D / 2 : D;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const int64_t qoff = (row_id * a.Hq + (int64_t)g * G + h) * kQWordsPerRow;
    const uint32_t* qp = reinterpret_cast<const uint32_t*>(a.q) + qoff;
    const uint32_t* qlp = reinterpret_cast<const uint32_t*>(W::kBf16 ? a.q_lo : a.q) + qoff;
#pragma unroll
    for (int j = 0; j < W::CPL * W::QC; ++j) wk.set_q(h, j, ld16(qp + wk.q_chunk(j) * 4), ld16(qlp + wk.q_chunk(j) * 4));
  }

  const int64_t lbase = (int64_t)(a.layer0 + l) * a.layer_elems;
  const T* kpool = reinterpret_cast<const T*>(a.k_pool) + lbase;
  const T* vpool = reinterpret_cast<const T*>(a.v_pool) + lbase;
  const int32_t* bt = a.block_tables + (int64_t)b * a.max_pages;
  SplitPages sp;
  sp.init(bt, kb / kPage, a.max_pages, wk.lane);
  wk.run(kb, k1, a.scale_log2, [&](int j, typename W::Row& rw) {
    const int32_t page = sp.page_of(j);
    const bool valid = page >= 0 && page < a.n_pages;
    rw.ok = valid && j >= k0;
    rw.lds = false;
    const int64_t roff = (((int64_t)(valid ? page : 0) * a.Hkv + g) * kPage + (j % kPage)) * D;
#pragma unroll
    for (int i = 0; i < W::CPL; ++i) rw.k[i] = ld16_stream(kpool + roff + (wk.tl + W::TL * i) * W::CH);
#pragma unroll
    for (int i = 0; i < W::CPL; ++i) rw.v[i] = ld16_stream(vpool + roff + (wk.tl + W::TL * i) * W::CH);
  }, [] {});

  __shared__ float s_acc[4][G][D];
  __shared__ float s_ml[4][G][2];
  wk.to_lds(s_acc, s_ml);
  __syncthreads();

  const int64_t part_base = (row_id * a.Hq + (int64_t)g * G) * a.n_split_max + s;  // head 0 of group
  for (int t = threadIdx.x; t < G * D; t += kThreads) {
    const int h = t / D;
    const int d = t - h * D;
    float m, lsum, o;
    wave_merge<G, D>(s_acc, s_ml, h, d, m, lsum, o);
    const int64_t pidx = part_base + (int64_t)h * a.n_split_max;
    a.part_acc[pidx * D + d] = o;
    if (d == 0) {
      a.part_ml[pidx * 2] = m;
      a.part_ml[pidx * 2 + 1] = lsum;
    }
  }
}

__global__ __launch_bounds__(kThreads) void attn_merge_kernel(const AttnArgs a) {
  int64_t w = blockIdx.x;                       // (layer, batch, row, q head)
  w /= a.Hq;
  const int r = (int)(w % a.rows); w /= a.rows;
  const int b = (int)(w % a.batch); w /= a.batch;
  const int l = (int)w;
  const int64_t row_head = blockIdx.x;
  float* out = a.out + row_head * a.D;
  const int ctx = a.ctx_lens[b];
  if (ctx < 0 || ctx > a.max_ctx_len) {
    for (int d = threadIdx.x; d < a.D; d += kThreads) out[d] = __int_as_float(0x7FC00000);
    return;
  }
  const int n_keys = ctx + r + 1;
  const int n_split = split_count(n_keys, window_start(layer_window(a, l), n_keys));
  const float* ml = a.part_ml + row_head * a.n_split_max * 2;
  const float* acc = a.part_acc + row_head * a.n_split_max * a.D;
  for (int d = threadIdx.x; d < a.D; d += kThreads) out[d] = combine_splits(ml, acc + d, a.D, n_split);
}

// ------------------------------------------------------------------------------------
// Decode: the split kernel rotates its queries from the raw input (angles in fp64 once per
// workgroup) and the last split's workgroup appends the new token's K/V for its KV head
// (written to the cache and kept in LDS for its own use).  A context that fits one split
// is finished in place; longer ones are combined by decode_merge_kernel in ascending split
// order.  (Combining in the last-arriving workgroup would need a device-scope release per
// workgroup, an L2 write-back on this chip that cost more than the second launch.)
template <typename T>
__device__ __forceinline__ void rotate_chunk(const uint4& va, const uint4& vb, bool first_half, int pair0,
                                             int pairing, const float* cs, float* out) {
  constexpr int E = Elem<T>::kPerVec;
  if (pairing == 0) {
    // va: this chunk, vb: its partner D/2 away; pair index pair0 + e
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float x = first_half ? Elem<T>::get(va, e) : Elem<T>::get(vb, e);   // first-half element
      float y = first_half ? Elem<T>::get(vb, e) : Elem<T>::get(va, e);   // second-half element
      rotate_pair(x, y, cs[2 * (pair0 + e)], cs[2 * (pair0 + e) + 1]);
      out[e] = first_half ? x : y;
    }
  } else {
#pragma unroll
    for (int e = 0; e < E; e += 2) {
      float x = Elem<T>::get(va, e), y = Elem<T>::get(va, e + 1);
      const int p = pair0 + (e >> 1);
      rotate_pair(x, y, cs[2 * p], cs[2 * p + 1]);
      out[e] = x;
      out[e + 1] = y;
    }
  }
}

template <typename T>
__device__ __forceinline__ uint4 pack_chunk(const float* x) {
  constexpr int E = Elem<T>::kPerVec;
  uint4 v = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int e = 0; e < E; ++e) Elem<T>::put(v, e, x[e]);
  return v;
}

// Rotated values of 16-byte chunk c of a raw row (pairing-aware), in fp32.
template <typename T, int D>
__device__ __forceinline__ void rotated_values(const T* raw_row, int c, int pairing, const float* cs, float* x) {
  constexpr int E = Elem<T>::kPerVec;
  constexpr int NCH = D / E;
  const uint4 va = ld16(raw_row + c * E);
  if (pairing == 0) {
    const bool first = c < NCH / 2;
    const int cp = first ? c + NCH / 2 : c - NCH / 2;
    const uint4 vb = ld16(raw_row + cp * E);
    rotate_chunk<T>(va, vb, first, (first ? c : cp) * E, 0, cs, x);
  } else {
    rotate_chunk<T>(va, va, true, c * E / 2, 1, cs, x);
  }
}

// Rotated 16-byte query chunk c of a raw row: for bf16 rows as the hi and lo parts of
// split_bf16, for fp32 rows the values themselves (lo unused).
template <typename T, int D>
__device__ __forceinline__ void rotated_query_chunk(const T* raw_row, int c, int pairing, const float* cs, uint4& hi,
                                                    uint4& lo) {
  constexpr int E = Elem<T>::kPerVec;
  float x[E];
  rotated_values<T, D>(raw_row, c, pairing, cs, x);
  if constexpr (sizeof(T) == 2) {
    uint32_t h[E], l[E];
#pragma unroll
    for (int e = 0; e < E; ++e) split_bf16(x[e], h[e], l[e]);
    hi = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    lo = make_uint4(l[0] | (l[1] << 16), l[2] | (l[3] << 16), l[4] | (l[5] << 16), l[6] | (l[7] << 16));
  } else {
    hi = pack_chunk<T>(x);
    lo = hi;
  }
}

// Chunk c of a storage row of type T (rotated or not) from a raw row of type R: the raw
// chunks it covers (two bf16 chunks per fp8 chunk), rounded once to T.
template <typename T, typename R, int D>
__device__ __forceinline__ uint4 storage_chunk(const R* raw_row, int c, bool rotate, int pairing, const float* cs) {
  constexpr int ET = Elem<T>::kPerVec, ER = Elem<R>::kPerVec, P = ET / ER;
  float x[ET];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    if (rotate) {
      rotated_values<R, D>(raw_row, c * P + p, pairing, cs, x + p * ER);
    } else {
      const uint4 v = ld16(raw_row + (c * P + p) * ER);
#pragma unroll
      for (int e = 0; e < ER; ++e) x[p * ER + e] = Elem<R>::get(v, e);
    }
  }
  uint32_t w[4];
  pack_words<T, ET>(x, w);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void decode_kernel(const DecodeArgs a) {
  using W = SplitWorker<T, D, G>;
  using R = typename W::QD;                         // raw input type (bf16 for fp8 caches)
  constexpr int NCH = W::NCH;                       // 16-byte chunks of a cache row
  constexpr int ER = Elem<R>::kPerVec;
  constexpr int NCHR = D / ER;                      // 16-byte chunks of a raw row
  // Sequence index fastest.  When the sequences share leading pages (a shared window,
  // shared_order), runs of 64 consecutive work items go to one XCD (workgroups are dealt
  // to the 8 XCDs in turn), so the sequences reading the same keys do so at about the same
  // time through one L2: 32 sequences over a shared 32k-token window decode 8 steps in
  // 212 instead of 367 ms.  Private pages keep the plain order, which measured 5% faster
  // there.  The arithmetic of a work item does not depend on the order.
  int64_t w = blockIdx.x;
  if (a.shared_order) {
    constexpr int64_t CH = 64;
    const int64_t full = (int64_t)gridDim.x / (8 * CH) * (8 * CH);
    if (w < full) {
      const int64_t g8 = w / 8;
      w = ((g8 / CH) * 8 + w % 8) * CH + g8 % CH;
    }
  }
  const int b = (int)(w % a.batch);        w /= a.batch;
  const int si = (int)(w % a.n_split_grid); w /= a.n_split_grid;
  const int g = (int)(w % a.Hkv);          w /= a.Hkv;
  const int l = (int)w;

  const int tid = threadIdx.x;
  constexpr int QCH = G * NCHR;                     // 16-byte chunks of the group's raw q
  constexpr int QPT = (QCH + kThreads - 1) / kThreads;
  const int64_t tok = (int64_t)l * a.batch + b;   // the step's raw row index

  // Requested before the context length is known, which they do not depend on: the
  // split's block-table entries, then the step's raw rows (the prologue waits for these
  // alone, the memory counter being in order; every thread loads one 16-byte chunk, indices
  // clamped; the new token's k and v are read by every split, used by the last).
  const int32_t* bt = a.block_tables + (int64_t)b * a.max_pages;
  const int win = layer_window(a, l);
  // the grid holds no shared split (the shared-split kernel's): a full-attention layer's
  // items start after them
  const int s = (win == 0 ? a.n_shared_split : 0) + si;
  SplitPages sp;
  if (win == 0) sp.init(bt, s * (kSplit / kPage), a.max_pages, tid & 63);   // split s = keys [512 s, ...)
  uint4 rq[QPT];
  const R* qraw = reinterpret_cast<const R*>(a.q_raw) + (tok * a.Hq + (int64_t)g * G) * D;
#pragma unroll
  for (int r = 0; r < QPT; ++r) rq[r] = ld16(qraw + min(tid + r * kThreads, QCH - 1) * ER);
  const R* kraw = reinterpret_cast<const R*>(a.k_raw) + (tok * a.Hkv + g) * D;
  const R* vraw = reinterpret_cast<const R*>(a.v_raw) + (tok * a.Hkv + g) * D;
  const uint4 rk = ld16(kraw + min(tid, NCHR - 1) * ER);
  const uint4 rv = ld16(vraw + min(tid, NCHR - 1) * ER);
  __builtin_amdgcn_sched_barrier(0);              // keep these loads ahead of the key rows

  const int ctx = a.ctx_lens[b];
  if (ctx < 0 || ctx > a.max_ctx_len) return;
  const int n_keys = ctx + 1;                     // the new token is key ctx
  const int lo = window_start(win, n_keys);
  const int n_split = split_count(n_keys, lo);
  if (s >= n_split) return;
  const int k0 = lo + s * kSplit;                 // the split's keys [k0, k1)
  const int k1 = min(k0 + kSplit, n_keys);
  const int kb = k0 & ~(kPage - 1);               // teams start at the page holding k0
  const bool last_split = s == n_split - 1;
  if (win != 0) sp.init(bt, kb / kPage, a.max_pages, tid & 63);

  __shared__ float cs[2 * kMaxHalfDim];
  __shared__ uint4 new_k[NCH], new_v[NCH];
  __shared__ uint4 raw_q[QCH], raw_k[NCHR], raw_v[NCHR];
  __shared__ float s_acc[4][G][D];
  __shared__ float s_ml[4][G][2];

  const int64_t lbase = (int64_t)(a.layer0 + l) * a.layer_elems;
  T* kpool = reinterpret_cast<T*>(a.k_pool) + lbase;
  T* vpool = reinterpret_cast<T*>(a.v_pool) + lbase;
  const int64_t pos = a.start_pos[b] + ctx;       // absolute position of the new token

  W wk;
  wk.init();
  wk.lds_k = new_k;
  wk.lds_v = new_v;

  // The new token (key ctx) is not in the cache yet when its row is requested: its slot's
  // old bytes are loaded like any row (in bounds, discarded) and the key is consumed from
  // LDS, so no branch depends on the key.
  auto load = [&](int j, typename W::Row& rw) {
    const int32_t page = sp.page_of(j);
    const bool valid = page >= 0 && page < a.n_pages;
    rw.lds = j == ctx;
    rw.ok = rw.lds || (valid && j >= k0);
    const int64_t roff = (((int64_t)(valid ? page : 0) * a.Hkv + g) * kPage + (j % kPage)) * D;
#pragma unroll
    for (int i = 0; i < W::CPL; ++i) rw.k[i] = ld16_stream(kpool + roff + (wk.tl + W::TL * i) * W::CH);
#pragma unroll
    for (int i = 0; i < W::CPL; ++i) rw.v[i] = ld16_stream(vpool + roff + (wk.tl + W::TL * i) * W::CH);
  };
  // runs while the first key rows are in flight: rotation table, the new token's K/V
  // (last split: rotated K, written to the cache and kept in LDS), the rotated queries
  auto prologue = [&] {
    for (int p = tid; p < D / 2; p += kThreads) {
      double sn, cn;
      sincos((double)pos * a.theta[p], &sn, &cn);
      cs[2 * p] = (float)cn;
      cs[2 * p + 1] = (float)sn;
    }
#pragma unroll
    for (int r = 0; r < QPT; ++r)
      if (tid + r * kThreads < QCH) raw_q[tid + r * kThreads] = rq[r];
    if (tid < NCHR) {
      raw_k[tid] = rk;
      raw_v[tid] = rv;
    }
    __syncthreads();
    // the new token's V in the cache dtype (every split: a row equal to key ctx is taken
    // from LDS when it is consumed, which only the last split does)
    for (int c = tid; c < NCH; c += kThreads)
      new_v[c] = storage_chunk<T, R, D>(reinterpret_cast<const R*>(raw_v), c, false, a.pairing, cs);
    if (last_split) {
      const int32_t page = sp.page_of(ctx);
      const bool ok = page >= 0 && page < a.n_pages;
      const int64_t roff = (((int64_t)(ok ? page : 0) * a.Hkv + g) * kPage + (ctx % kPage)) * D;
      for (int c = tid; c < NCH; c += kThreads) {
        const uint4 kc = storage_chunk<T, R, D>(reinterpret_cast<const R*>(raw_k), c, true, a.pairing, cs);
        new_k[c] = kc;
        if (ok) {
          st16(kpool + roff + c * W::CH, kc);
          st16(vpool + roff + c * W::CH, new_v[c]);       // written by this thread above
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int j = 0; j < W::CPL * W::QC; ++j) {
        uint4 hi, lo;
        rotated_query_chunk<R, D>(reinterpret_cast<const R*>(raw_q) + h * D, wk.q_chunk(j), a.pairing, cs, hi, lo);
        wk.set_q(h, j, hi, lo);
      }
  };
  wk.run(kb, k1, a.scale_log2, load, prologue);

  wk.to_lds(s_acc, s_ml);
  __syncthreads();

  const int64_t head0 = tok * a.Hq + (int64_t)g * G;     // output row of head 0 of the group
  if (n_split == 1) {
    for (int t = tid; t < G * D; t += kThreads) {
      const int h = t / D, d = t - (t / D) * D;
      alignas(8) float ml[2];
      float o;
      wave_merge<G, D>(s_acc, s_ml, h, d, ml[0], ml[1], o);
      a.out[(head0 + h) * D + d] = combine_splits(ml, &o, 0, 1);
    }
    return;
  }

  // publish this split's partial; decode_merge_kernel combines the splits
  for (int t = tid; t < G * D; t += kThreads) {
    const int h = t / D, d = t - (t / D) * D;
    float m, lsum, o;
    wave_merge<G, D>(s_acc, s_ml, h, d, m, lsum, o);
    const int64_t pidx = (head0 + h) * a.n_split_max + s;
    a.part_acc[pidx * D + d] = o;
    if (d == 0) {
      a.part_ml[pidx * 2] = m;
      a.part_ml[pidx * 2 + 1] = lsum;
    }
  }
}

// Combine the split partials of every (layer, sequence, query head) row whose context
// needed more than one split, in ascending split order.
__global__ __launch_bounds__(kThreads) void decode_merge_kernel(const DecodeArgs a) {
  const int64_t row_head = blockIdx.x;            // (layer, batch, q head)
  const int b = (int)((row_head / a.Hq) % a.batch);
  const int l = (int)(row_head / ((int64_t)a.Hq * a.batch));
  constexpr int U = 16;
  if (a.n_split_max <= U && a.D <= kThreads) {
    // One memory round trip: the partials of every split the workspace holds are requested
    // together with the context length (in bounds; those of splits the row does not use
    // are not added), then combined exactly as combine_splits does.
    const float* ml = a.part_ml + row_head * a.n_split_max * 2;
    const float* acc = a.part_acc + row_head * a.n_split_max * a.D;
    const int d = min((int)threadIdx.x, a.D - 1);
    float2 pv[U];
    float av[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = min(u, a.n_split_max - 1);
      pv[u] = *reinterpret_cast<const float2*>(ml + 2 * s);
      av[u] = acc[s * a.D + d];
    }
    const int ctx = a.ctx_lens[b];
    if (ctx < 0 || ctx > a.max_ctx_len) return;
    const int win = layer_window(a, l);
    const int n_split = split_count(ctx + 1, window_start(win, ctx + 1));
    if (n_split == 1 && !(win == 0 && a.n_shared_split > 0)) return;   // written by the split kernel
    float m = -INFINITY;
#pragma unroll
    for (int u = 0; u < U; ++u) m = (u < n_split) ? fmaxf(m, pv[u].x) : m;
    float lsum = 0.0f, o = 0.0f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float f = merge_factor(pv[u].x, m);
      const bool in = u < n_split;
      lsum = in ? fmaf(pv[u].y, f, lsum) : lsum;
      o = in ? fmaf(av[u], f, o) : o;
    }
    if ((int)threadIdx.x < a.D) a.out[row_head * a.D + threadIdx.x] = o / lsum;
    return;
  }
  const int ctx = a.ctx_lens[b];
  if (ctx < 0 || ctx > a.max_ctx_len) return;
  const int win = layer_window(a, l);
  const int n_split = split_count(ctx + 1, window_start(win, ctx + 1));
  if (n_split == 1 && !(win == 0 && a.n_shared_split > 0)) return;     // written by the split kernel
  const float* ml = a.part_ml + row_head * a.n_split_max * 2;
  const float* acc = a.part_acc + row_head * a.n_split_max * a.D;
  constexpr int kLdsSplits = 2048;
  if (n_split <= kLdsSplits) {
    // Many splits (long contexts, shared windows): the (reference, sum) pairs are staged in
    // LDS by the whole workgroup in one round trip, and each lane requests 16 splits' values
    // at a time; the arithmetic and its order are combine_splits' own.
    __shared__ float s_ml[2 * kLdsSplits];
    for (int t = threadIdx.x; t < 2 * n_split; t += kThreads) s_ml[t] = ml[t];
    __syncthreads();
    float m = -INFINITY;
    for (int s = 0; s < n_split; ++s) m = fmaxf(m, s_ml[2 * s]);
    constexpr int U = 16;
    for (int d = threadIdx.x; d < a.D; d += kThreads) {
      float lsum = 0.0f, o = 0.0f;
      for (int s0 = 0; s0 < n_split; s0 += U) {
        float av[U];
#pragma unroll
        for (int u = 0; u < U; ++u) av[u] = acc[min(s0 + u, n_split - 1) * a.D + d];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int s = min(s0 + u, n_split - 1);
          const float f = merge_factor(s_ml[2 * s], m);
          const bool in = s0 + u < n_split;
          lsum = in ? fmaf(s_ml[2 * s + 1], f, lsum) : lsum;
          o = in ? fmaf(av[u], f, o) : o;
        }
      }
      a.out[row_head * a.D + d] = o / lsum;
    }
    return;
  }
  for (int d = threadIdx.x; d < a.D; d += kThreads)
    a.out[row_head * a.D + d] = combine_splits(ml, acc + d, a.D, n_split);
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

template <typename T, int D>
hipError_t launch_decode_g(const DecodeArgs& a, hipStream_t stream) {
  const int64_t n_blocks = (int64_t)a.n_layers * a.batch * a.Hkv * a.n_split_grid;
  switch (a.group) {
    case 1: decode_kernel<T, D, 1><<<dim3((unsigned)n_blocks), kThreads, 0, stream>>>(a); break;
    case 2: decode_kernel<T, D, 2><<<dim3((unsigned)n_blocks), kThreads, 0, stream>>>(a); break;
    case 4: decode_kernel<T, D, 4><<<dim3((unsigned)n_blocks), kThreads, 0, stream>>>(a); break;
    case 8: decode_kernel<T, D, 8><<<dim3((unsigned)n_blocks), kThreads, 0, stream>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_decode_d(const DecodeArgs& a, hipStream_t stream) {
  switch (a.D) {
    case 64: return launch_decode_g<T, 64>(a, stream);
    case 128: return launch_decode_g<T, 128>(a, stream);
    case 256: return launch_decode_g<T, 256>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

// Suffix prefill over shared pages: each row's two partials (the shared pages, from the
// shared-split mode of the MFMA kernel; the sequence's own keys, from its per-sequence mode)
// combined in that order, on full-attention layers.
__global__ __launch_bounds__(kThreads) void prefill_combine_kernel(const PrefillArgs a, int64_t n_rows) {
  // a workgroup per (layer, sequence, chunk row, query head), grid-strided
  for (int64_t row_head = blockIdx.x; row_head < n_rows; row_head += gridDim.x) {
    const int b = (int)((row_head / ((int64_t)a.Hq * a.chunk)) % a.batch);
    const int l = (int)(row_head / ((int64_t)a.Hq * a.chunk * a.batch));
    if (layer_window(a, l) != 0) continue;        // written by the per-sequence kernel
    const int ctx = a.ctx_lens[b];
    if (ctx < 0 || ctx > a.max_ctx_len) continue;
    const float* ml = a.part_ml + row_head * a.n_split_max * 2;
    const float* acc = a.part_acc + row_head * a.n_split_max * a.D;
    for (int d = threadIdx.x; d < a.D; d += kThreads)
      a.out[row_head * a.D + d] = combine_splits<2>(ml, acc + d, a.D, a.n_split_max);
  }
}

}  // namespace

hipError_t launch_attn_valu(const AttnArgs& a, int dtype, hipStream_t stream) {
  hipError_t e = dtype == kDtypeBf16  ? launch_partial_d<uint16_t>(a, stream)
                 : dtype == kDtypeFp8 ? launch_partial_d<uint8_t>(a, stream)
                                      : launch_partial_d<float>(a, stream);
  if (e != hipSuccess) return e;
  const int64_t n_rows = (int64_t)a.n_layers * a.batch * a.rows * a.Hq;
  attn_merge_kernel<<<dim3((unsigned)n_rows), kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_prefill_combine(const PrefillArgs& a, hipStream_t stream) {
  const int64_t n_rows = (int64_t)a.n_layers * a.batch * a.chunk * a.Hq;
  if (n_rows <= 0) return hipSuccess;
  const unsigned n_wg = (unsigned)std::min<int64_t>(n_rows, int64_t(1) << 22);   // 2^30 threads at most
  prefill_combine_kernel<<<dim3(n_wg), kThreads, 0, stream>>>(a, n_rows);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs& a, int dtype, hipStream_t stream) {
  hipError_t e = dtype == kDtypeBf16  ? launch_decode_d<uint16_t>(a, stream)
                 : dtype == kDtypeFp8 ? launch_decode_d<uint8_t>(a, stream)
                                      : launch_decode_d<float>(a, stream);
  if (e != hipSuccess) return e;
  const int64_t n_rows = (int64_t)a.n_layers * a.batch * a.Hq;
  decode_merge_kernel<<<dim3((unsigned)n_rows), kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace kvg
