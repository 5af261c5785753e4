// C ABI of libkvg: argument validation, workspace carving and kernel launches.
// Every check runs on the host before anything is enqueued.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>

#include "kvg.h"
#include "kvg_launch.h"

namespace {

using kvg::kPage;
using kvg::kSplit;

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

size_t elem_bytes(const kvg_cache* c) { return c->dtype == KVG_BF16 ? 2 : c->dtype == KVG_FP8_E4M3 ? 1 : 4; }

// bytes of one raw q/k/v element (an fp8 cache takes bf16 inputs) and of a rotated query
// in the attention workspace (bf16 for bf16 and fp8 caches)
size_t raw_bytes(const kvg_cache* c) { return c->dtype == KVG_F32 ? 4 : 2; }

int check_cache(const kvg_cache* c) {
  if (c == nullptr || c->k_pool == nullptr || c->v_pool == nullptr) return KVG_E_INVAL;
  if (c->dtype != KVG_F32 && c->dtype != KVG_BF16 && c->dtype != KVG_FP8_E4M3) return KVG_E_DTYPE;
  if (c->n_layers <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->n_pages <= 0) return KVG_E_SHAPE;
  if (c->n_pages > INT32_MAX) return KVG_E_SHAPE;
  if (c->head_dim != 64 && c->head_dim != 128 && c->head_dim != 256) return KVG_E_SHAPE;
  if (c->page_size != kPage) return KVG_E_SHAPE;
  if (c->n_q_heads % c->n_kv_heads != 0) return KVG_E_SHAPE;
  const int g = c->n_q_heads / c->n_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8) return KVG_E_SHAPE;
  if (c->layer_window != nullptr)
    for (int l = 0; l < c->n_layers; ++l)
      if (c->layer_window[l] < 0) return KVG_E_INVAL;
  return KVG_OK;
}

// Windows of layers [layer0, layer0 + n_layers) as a launch carries them (all zero when none
// is windowed); KVG_E_SHAPE when a windowed call spans more layers than a launch carries.
int fill_windows(const kvg_cache* c, int32_t layer0, int32_t n_layers, int32_t* dst) {
  std::memset(dst, 0, sizeof(int32_t) * kvg::kMaxWindowLayers);
  if (c->layer_window == nullptr) return KVG_OK;
  bool any = false;
  for (int l = 0; l < n_layers; ++l) any = any || c->layer_window[layer0 + l] != 0;
  if (!any) return KVG_OK;
  if (n_layers > kvg::kMaxWindowLayers) return KVG_E_SHAPE;
  for (int l = 0; l < n_layers; ++l) dst[l] = c->layer_window[layer0 + l];
  return KVG_OK;
}

int check_rope(const kvg_rope* r) {
  if (r == nullptr || !(r->base > 0.0) || !std::isfinite(r->base)) return KVG_E_INVAL;
  if (r->pairing != KVG_ROPE_HALF && r->pairing != KVG_ROPE_INTERLEAVED) return KVG_E_INVAL;
  if (r->reserved != 0) return KVG_E_INVAL;
  return KVG_OK;
}

int check_layers(const kvg_cache* c, int32_t layer0, int32_t n_layers) {
  if (layer0 < 0 || n_layers <= 0 || layer0 + (int64_t)n_layers > c->n_layers) return KVG_E_SHAPE;
  return KVG_OK;
}

int check_seqs(const kvg_cache* c, const kvg_seqs* s, int32_t chunk) {
  if (s == nullptr || s->block_tables == nullptr || s->ctx_lens == nullptr || s->start_pos == nullptr)
    return KVG_E_INVAL;
  if (s->batch <= 0 || s->max_pages <= 0 || s->max_ctx_len < 0 || chunk <= 0 || s->shared_tokens < 0 ||
      (int64_t)s->shared_tokens > (int64_t)s->max_pages * c->page_size)
    return KVG_E_INVAL;
  if ((int64_t)s->max_ctx_len + chunk > (int64_t)s->max_pages * c->page_size) return KVG_E_CAPACITY;
  return KVG_OK;
}

int64_t layer_elems(const kvg_cache* c) {
  return c->n_pages * c->n_kv_heads * (int64_t)c->page_size * c->head_dim;
}

int n_split_max(const kvg_seqs* s, int32_t chunk) {
  return (int)(((int64_t)s->max_ctx_len + chunk + kSplit - 1) / kSplit);
}

// Workspace of the vector-ALU attention path: rotated queries (fp32, or bf16 hi and lo
// planes for bf16 and fp8 caches), split partials.
struct ValuWs {
  size_t q, q_plane, acc, ml, total;
};

ValuWs valu_ws(const kvg_cache* c, const kvg_seqs* s, int32_t n_layers, int32_t rows) {
  ValuWs w;
  const size_t nrow_heads = (size_t)n_layers * s->batch * rows * c->n_q_heads;
  const size_t ns = (size_t)n_split_max(s, rows);
  w.q_plane = align_up(nrow_heads * c->head_dim * raw_bytes(c));
  w.q = c->dtype == KVG_F32 ? w.q_plane : 2 * w.q_plane;
  w.acc = align_up(nrow_heads * ns * c->head_dim * sizeof(float));
  w.ml = align_up(nrow_heads * ns * 2 * sizeof(float));
  w.total = w.q + w.acc + w.ml;
  return w;
}

kvg::AppendArgs append_args(const kvg_cache* c, const kvg_seqs* s, const kvg_rope* r, int32_t layer0,
                            int32_t n_layers, int32_t chunk, const void* k_raw, const void* v_raw) {
  kvg::AppendArgs a;
  std::memset(&a, 0, sizeof(a));
  a.k_pool = c->k_pool;
  a.v_pool = c->v_pool;
  a.layer_elems = layer_elems(c);
  a.n_pages = c->n_pages;
  a.block_tables = s->block_tables;
  a.ctx_lens = s->ctx_lens;
  a.start_pos = s->start_pos;
  a.k_raw = k_raw;
  a.v_raw = v_raw;
  a.Hq = c->n_q_heads;
  a.Hkv = c->n_kv_heads;
  a.D = c->head_dim;
  a.layer0 = layer0;
  a.n_layers = n_layers;
  a.batch = s->batch;
  a.chunk = chunk;
  a.max_pages = s->max_pages;
  a.max_ctx_len = s->max_ctx_len;
  a.pairing = r->pairing;
  // layers per workgroup: enough workgroups to fill the chip, fewer sincos recomputations
  const int64_t tokens = (int64_t)s->batch * chunk;
  int64_t lpb = ((int64_t)n_layers * tokens + 8191) / 8192;
  if (lpb < 1) lpb = 1;
  if (lpb > n_layers) lpb = n_layers;
  a.layers_per_block = (int32_t)lpb;
  for (int i = 0; i < c->head_dim / 2; ++i) a.theta[i] = std::pow(r->base, -2.0 * i / c->head_dim);
  return a;
}

int hip_status(hipError_t e) { return e == hipSuccess ? KVG_OK : KVG_E_HIP; }

// A launch of `wgs` workgroups of `threads` threads fits the dispatch limits (grid size in
// threads below 2^32).  Every launch of a call is checked before the first one is enqueued.
bool fits_grid(int64_t wgs, int threads) { return wgs >= 0 && wgs * (int64_t)threads <= (int64_t)UINT32_MAX; }

// The append's grid: (batch * chunk) x layer groups of 256 threads.
bool append_fits(const kvg_seqs* s, int32_t chunk) { return fits_grid((int64_t)s->batch * chunk, 256); }

int check_raw(const void* k_raw, const void* v_raw) {
  return (k_raw == nullptr || v_raw == nullptr) ? KVG_E_INVAL : KVG_OK;
}

// Shared body of the vector-ALU attention calls: append, rotate queries, partials, merge.
int attn_valu(const kvg_cache* c, const kvg_seqs* s, const kvg_rope* r, int32_t layer0, int32_t n_layers,
              int32_t rows, const void* q_raw, const void* k_raw, const void* v_raw, float scale,
              float* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  const ValuWs w = valu_ws(c, s, n_layers, rows);
  if (ws == nullptr || ws_bytes < w.total) return KVG_E_WORKSPACE;
  const int64_t n_blocks = (int64_t)n_layers * s->batch * rows * c->n_kv_heads * n_split_max(s, rows);
  const int64_t n_rows = (int64_t)n_layers * s->batch * rows * c->n_q_heads;
  if (!fits_grid(n_blocks, 256) || !fits_grid(n_rows, 256) || !append_fits(s, rows)) return KVG_E_SHAPE;
  char* base = static_cast<char*>(ws);
  void* q = base;
  float* acc = reinterpret_cast<float*>(base + w.q);
  float* ml = reinterpret_cast<float*>(base + w.q + w.acc);

  void* q_lo = c->dtype == KVG_F32 ? nullptr : base + w.q_plane;
  kvg::AppendArgs ap = append_args(c, s, r, layer0, n_layers, rows, k_raw, v_raw);
  ap.q_raw = q_raw;
  ap.q_out = q;
  ap.q_out_lo = q_lo;
  ap.q_out_bf16 = c->dtype != KVG_F32;
  int st = hip_status(kvg::launch_append(ap, c->dtype, stream));
  if (st != KVG_OK) return st;

  kvg::AttnArgs a;
  std::memset(&a, 0, sizeof(a));
  a.k_pool = c->k_pool;
  a.v_pool = c->v_pool;
  a.layer_elems = layer_elems(c);
  a.n_pages = c->n_pages;
  a.block_tables = s->block_tables;
  a.ctx_lens = s->ctx_lens;
  a.q = q;
  a.q_lo = q_lo;
  a.part_acc = acc;
  a.part_ml = ml;
  a.out = out;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.Hq = c->n_q_heads;
  a.Hkv = c->n_kv_heads;
  a.D = c->head_dim;
  a.group = c->n_q_heads / c->n_kv_heads;
  a.layer0 = layer0;
  a.n_layers = n_layers;
  a.batch = s->batch;
  a.rows = rows;
  a.max_pages = s->max_pages;
  a.max_ctx_len = s->max_ctx_len;
  a.n_split_max = n_split_max(s, rows);
  fill_windows(c, layer0, n_layers, a.window);
  return hip_status(kvg::launch_attn_valu(a, c->dtype, stream));
}

// Workspace of the decode kernels: the split partials.
// bf16 and fp8 caches with up to 4 query heads per KV head prefill on MFMA; others on the
// VALU path.
bool use_mfma(const kvg_cache* c) {
  return (c->dtype == KVG_BF16 || c->dtype == KVG_FP8_E4M3) && c->n_q_heads / c->n_kv_heads <= 4;
}

// Decode splits served by the shared-split kernel: the whole 512-key splits inside the
// leading pages every sequence shares (kvg_seqs.shared_tokens), when several sequences
// share them and the cache takes the MFMA path; 0 otherwise.
int shared_splits(const kvg_cache* c, const kvg_seqs* s) {
  if (s->shared_tokens <= 0 || s->batch < 2 || !use_mfma(c)) return 0;
  return std::min(s->shared_tokens / kSplit, n_split_max(s, 1));
}

// Splits per (layer, sequence, KV head) in the decode kernel's grid: every split, less the
// shared ones of full-attention layers (the shared-split kernel's), but at least as many as
// a windowed layer of the range can have (its splits count from the window's first key).
int decode_grid_splits(const kvg_cache* c, const kvg_seqs* s, int32_t layer0, int32_t n_layers) {
  const int n_split = n_split_max(s, 1);
  const int shared = shared_splits(c, s);
  if (shared == 0) return n_split;
  int grid = n_split - shared;
  if (c->layer_window != nullptr)
    for (int l = 0; l < n_layers; ++l) {
      const int64_t W = c->layer_window[layer0 + l];
      if (W > 0) grid = std::max<int64_t>(grid, std::min<int64_t>(n_split, (W + kSplit - 1) / kSplit));
    }
  return grid;
}

struct DecodeWs {
  size_t ml, acc, q, total;
};

// Split partials, and the rotated bf16 queries of the shared-split kernel when it runs.
DecodeWs decode_ws(const kvg_cache* c, const kvg_seqs* s, int32_t n_layers) {
  DecodeWs w;
  const size_t ns = (size_t)n_split_max(s, 1);
  const size_t heads = (size_t)n_layers * s->batch * c->n_q_heads;
  w.ml = align_up(heads * ns * 2 * sizeof(float));
  w.acc = align_up(heads * ns * c->head_dim * sizeof(float));
  w.q = shared_splits(c, s) > 0 ? 2 * align_up(heads * c->head_dim * 2) : 0;   // hi and lo planes
  w.total = w.ml + w.acc + w.q;
  return w;
}

// One plane of rotated bf16 queries (the workspace holds a hi and a lo plane); with shared
// pages also two partials per (row, head).
size_t mfma_q_plane(const kvg_cache* c, const kvg_seqs* s, int32_t n_layers, int32_t chunk) {
  return align_up((size_t)n_layers * s->batch * chunk * c->n_q_heads * c->head_dim * 2);
}
size_t mfma_q_bytes(const kvg_cache* c, const kvg_seqs* s, int32_t n_layers, int32_t chunk) {
  return 2 * mfma_q_plane(c, s, n_layers, chunk);
}

// Rows per head of one q-tile of the MFMA prefill kernel.
int prefill_tile_rows(const kvg_cache* c) {
  return 32 * kvg::prefill_mfma_waves(c->head_dim) / (c->n_q_heads / c->n_kv_heads);
}

// Keys of the shared pages a suffix prefill attends once for the batch: only when the chunk
// is shorter than one q-tile (each sequence's tile is then partly empty, and the batch's
// rows packed together read every shared page fewer times); 0 otherwise.
int prefill_shared_keys(const kvg_cache* c, const kvg_seqs* s, int32_t chunk) {
  return chunk < prefill_tile_rows(c) ? shared_splits(c, s) * kSplit : 0;
}

size_t mfma_ws(const kvg_cache* c, const kvg_seqs* s, int32_t n_layers, int32_t chunk) {
  const size_t rows = (size_t)n_layers * s->batch * chunk * c->n_q_heads;
  const size_t part = prefill_shared_keys(c, s, chunk) > 0 ? align_up(rows * 2 * 2 * sizeof(float)) +
                                                                 align_up(rows * 2 * c->head_dim * sizeof(float))
                                                           : 0;
  return mfma_q_bytes(c, s, n_layers, chunk) + part;
}

// MFMA prefill: append (queries rotated to bf16 into the workspace), then the attention.
int attn_mfma(const kvg_cache* c, const kvg_seqs* s, const kvg_rope* r, int32_t layer0, int32_t n_layers,
              int32_t chunk, const void* q_raw, const void* k_raw, const void* v_raw, float scale, float* out,
              void* ws, size_t ws_bytes, hipStream_t stream) {
  if (ws == nullptr || ws_bytes < mfma_ws(c, s, n_layers, chunk)) return KVG_E_WORKSPACE;
  const int group = c->n_q_heads / c->n_kv_heads;
  const int bm = prefill_tile_rows(c);
  const int n_qt = (chunk + bm - 1) / bm;
  const int64_t n_wg = (int64_t)n_layers * s->batch * c->n_kv_heads * n_qt;
  const int threads = 64 * kvg::prefill_mfma_waves(c->head_dim);
  if (!fits_grid(n_wg, threads) || !append_fits(s, chunk)) return KVG_E_SHAPE;
  if (prefill_shared_keys(c, s, chunk) > 0) {
    const int64_t sh_waves = ((int64_t)s->batch * chunk + 31) / 32 * group;
    const int64_t sh_wg = (int64_t)n_layers * c->n_kv_heads * ((sh_waves + kvg::prefill_mfma_waves(c->head_dim) - 1) /
                                                               kvg::prefill_mfma_waves(c->head_dim));
    if (!fits_grid(sh_wg, threads)) return KVG_E_SHAPE;   // the combine launch is grid-strided
  }
  uint16_t* q_lo = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + mfma_q_plane(c, s, n_layers, chunk));
  kvg::AppendArgs ap = append_args(c, s, r, layer0, n_layers, chunk, k_raw, v_raw);
  ap.q_raw = q_raw;
  ap.q_out = ws;
  ap.q_out_lo = q_lo;
  ap.q_out_bf16 = 1;
  int st = hip_status(kvg::launch_append(ap, c->dtype, stream));
  if (st != KVG_OK) return st;
  kvg::PrefillArgs a;
  std::memset(&a, 0, sizeof(a));
  a.k_pool = c->k_pool;
  a.v_pool = c->v_pool;
  a.layer_elems = layer_elems(c);
  a.n_pages = c->n_pages;
  a.block_tables = s->block_tables;
  a.ctx_lens = s->ctx_lens;
  a.q = static_cast<const uint16_t*>(ws);
  a.q_lo = q_lo;
  a.out = out;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.Hq = c->n_q_heads;
  a.Hkv = c->n_kv_heads;
  a.D = c->head_dim;
  a.group = group;
  a.layer0 = layer0;
  a.n_layers = n_layers;
  a.batch = s->batch;
  a.chunk = chunk;
  a.max_pages = s->max_pages;
  a.max_ctx_len = s->max_ctx_len;
  a.n_qt = n_qt;
  fill_windows(c, layer0, n_layers, a.window);
  const int shared_keys = prefill_shared_keys(c, s, chunk);
  if (shared_keys == 0) return hip_status(kvg::launch_prefill_mfma(a, c->dtype, stream));
  // Shared pages (kvg_seqs.shared_tokens): on full-attention layers the rows' attention over
  // keys [0, shared_keys) is computed once per page for the whole batch (shared-split mode,
  // partial slot 0) and over their own keys by the per-sequence kernel (slot 1); the two
  // partials are then combined.
  const size_t rows = (size_t)n_layers * s->batch * chunk * c->n_q_heads;
  char* base = static_cast<char*>(ws) + mfma_q_bytes(c, s, n_layers, chunk);
  a.part_ml = reinterpret_cast<float*>(base);
  a.part_acc = reinterpret_cast<float*>(base + align_up(rows * 2 * 2 * sizeof(float)));
  a.n_split_max = 2;
  kvg::PrefillArgs sh = a;
  sh.n_shared_split = 1;
  sh.shared_keys = shared_keys;
  const int waves = (int)(((int64_t)s->batch * chunk + 31) / 32) * group;   // 32 rows of one head per wave
  const int nw = kvg::prefill_mfma_waves(c->head_dim);
  sh.n_qt = (waves + nw - 1) / nw;
  st = hip_status(kvg::launch_shared_splits(sh, c->dtype, stream));
  if (st != KVG_OK) return st;
  a.key_lo = shared_keys;
  a.part_slot = 1;
  st = hip_status(kvg::launch_prefill_mfma(a, c->dtype, stream));
  if (st != KVG_OK) return st;
  return hip_status(kvg::launch_prefill_combine(a, stream));
}

int check_attn(const kvg_cache* c, const kvg_seqs* s, const kvg_rope* r, int32_t layer0, int32_t n_layers,
               int32_t rows, const void* q_raw, const void* k_raw, const void* v_raw, float scale, float* out) {
  int st = check_cache(c);
  if (st != KVG_OK) return st;
  if ((st = check_rope(r)) != KVG_OK) return st;
  if ((st = check_layers(c, layer0, n_layers)) != KVG_OK) return st;
  if ((st = check_seqs(c, s, rows)) != KVG_OK) return st;
  if (q_raw == nullptr || out == nullptr || check_raw(k_raw, v_raw) != KVG_OK) return KVG_E_INVAL;
  if (!(scale > 0.0f) || !std::isfinite(scale)) return KVG_E_INVAL;
  int32_t w[kvg::kMaxWindowLayers];
  return fill_windows(c, layer0, n_layers, w);
}

}  // namespace

extern "C" {

const char* kvg_version(void) { return "kvg 0.1.0 hip gfx950"; }

const char* kvg_status_str(int status) {
  switch (status) {
    case KVG_OK: return "ok";
    case KVG_E_INVAL: return "invalid argument";
    case KVG_E_SHAPE: return "shape mismatch or unsupported geometry";
    case KVG_E_DTYPE: return "dtype mismatch or unsupported dtype";
    case KVG_E_POSITION: return "graft position differs from the block's own position";
    case KVG_E_CAPACITY: return "block table too short";
    case KVG_E_ALIGN: return "block start not page aligned";
    case KVG_E_CORRUPT: return "artifact header inconsistent or payload differs from its digest";
    case KVG_E_HIP: return "HIP runtime error";
    case KVG_E_WORKSPACE: return "workspace too small";
    default: return "unknown status";
  }
}

size_t kvg_payload_bytes(const kvg_cache* cache, int32_t n_tokens) {
  if (check_cache(cache) != KVG_OK || n_tokens <= 0) return 0;
  const size_t pages = (size_t)(n_tokens + cache->page_size - 1) / cache->page_size;
  return (size_t)cache->n_layers * 2 * pages * cache->n_kv_heads * cache->page_size * cache->head_dim *
         elem_bytes(cache);
}

int kvg_artifact_header_init(const kvg_cache* cache, int32_t n_tokens, int64_t own_pos, const kvg_rope* rope,
                             kvg_artifact_hdr* hdr) {
  int st = check_cache(cache);
  if (st != KVG_OK) return st;
  if ((st = check_rope(rope)) != KVG_OK) return st;
  if (hdr == nullptr || n_tokens <= 0) return KVG_E_INVAL;
  std::memset(hdr, 0, sizeof(*hdr));
  hdr->magic = KVG_ARTIFACT_MAGIC;
  hdr->version = KVG_ARTIFACT_VERSION;
  hdr->dtype = cache->dtype;
  hdr->n_layers = cache->n_layers;
  hdr->n_kv_heads = cache->n_kv_heads;
  hdr->head_dim = cache->head_dim;
  hdr->page_size = cache->page_size;
  hdr->n_tokens = n_tokens;
  hdr->own_pos = own_pos;
  hdr->rope_base = rope->base;
  hdr->rope_pairing = rope->pairing;
  hdr->payload_bytes = kvg_payload_bytes(cache, n_tokens);
  return KVG_OK;
}

int kvg_append(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope, int32_t layer0,
               int32_t n_layers, int32_t chunk_len, const void* k_raw, const void* v_raw, void* stream) {
  int st = check_cache(cache);
  if (st != KVG_OK) return st;
  if ((st = check_rope(rope)) != KVG_OK) return st;
  if ((st = check_layers(cache, layer0, n_layers)) != KVG_OK) return st;
  if ((st = check_seqs(cache, seqs, chunk_len)) != KVG_OK) return st;
  if ((st = check_raw(k_raw, v_raw)) != KVG_OK) return st;
  if (!append_fits(seqs, chunk_len)) return KVG_E_SHAPE;
  kvg::AppendArgs a = append_args(cache, seqs, rope, layer0, n_layers, chunk_len, k_raw, v_raw);
  return hip_status(kvg::launch_append(a, cache->dtype, static_cast<hipStream_t>(stream)));
}

int kvg_deposit(const kvg_cache* cache, const int32_t* block_table, int32_t table_len, int32_t first_token,
                int32_t n_tokens, void* payload, void* stream) {
  int st = check_cache(cache);
  if (st != KVG_OK) return st;
  if (block_table == nullptr || payload == nullptr || n_tokens <= 0 || first_token < 0 || table_len <= 0)
    return KVG_E_INVAL;
  if (first_token % cache->page_size != 0) return KVG_E_ALIGN;
  const int32_t n_pages = (n_tokens + cache->page_size - 1) / cache->page_size;
  if ((int64_t)first_token / cache->page_size + n_pages > table_len) return KVG_E_CAPACITY;
  kvg::CopyArgs a;
  std::memset(&a, 0, sizeof(a));
  a.k_pool = cache->k_pool;
  a.v_pool = cache->v_pool;
  a.page_bytes = (int64_t)cache->n_kv_heads * cache->page_size * cache->head_dim * elem_bytes(cache);
  a.layer_bytes = cache->n_pages * a.page_bytes;
  a.n_pages = cache->n_pages;
  a.block_table = block_table;
  a.payload = payload;
  a.first_page = first_token / cache->page_size;
  a.n_block_pages = n_pages;
  a.n_tokens = n_tokens;
  a.n_layers = cache->n_layers;
  a.row_bytes = cache->head_dim * (int)elem_bytes(cache);
  a.Hkv = cache->n_kv_heads;
  a.D = cache->head_dim;
  if (!fits_grid(kvg::copy_workgroups(a, cache->dtype), 256)) return KVG_E_SHAPE;
  return hip_status(kvg::launch_deposit(a, static_cast<hipStream_t>(stream)));
}

int kvg_graft(const kvg_cache* cache, const kvg_artifact_hdr* hdr, const void* payload,
              const int32_t* block_table, int32_t table_len, int32_t first_token, int64_t target_pos,
              int32_t flags, void* stream) {
  int st = check_cache(cache);
  if (st != KVG_OK) return st;
  if (hdr == nullptr || payload == nullptr || block_table == nullptr || first_token < 0 || table_len <= 0)
    return KVG_E_INVAL;
  if (hdr->magic != KVG_ARTIFACT_MAGIC || hdr->version != KVG_ARTIFACT_VERSION || hdr->n_tokens <= 0)
    return KVG_E_CORRUPT;
  if (hdr->dtype != cache->dtype) return KVG_E_DTYPE;
  if (hdr->n_layers != cache->n_layers || hdr->n_kv_heads != cache->n_kv_heads ||
      hdr->head_dim != cache->head_dim || hdr->page_size != cache->page_size)
    return KVG_E_SHAPE;
  if (hdr->payload_bytes != kvg_payload_bytes(cache, hdr->n_tokens)) return KVG_E_CORRUPT;
  if (hdr->rope_pairing != KVG_ROPE_HALF && hdr->rope_pairing != KVG_ROPE_INTERLEAVED) return KVG_E_CORRUPT;
  if (!(hdr->rope_base > 0.0) || !std::isfinite(hdr->rope_base)) return KVG_E_CORRUPT;
  if (first_token % cache->page_size != 0) return KVG_E_ALIGN;
  const int32_t n_pages = (hdr->n_tokens + cache->page_size - 1) / cache->page_size;
  if ((int64_t)first_token / cache->page_size + n_pages > table_len) return KVG_E_CAPACITY;
  const int64_t d = target_pos - hdr->own_pos;
  if (d != 0 && !(flags & KVG_GRAFT_ALLOW_RELOCATE)) return KVG_E_POSITION;

  kvg::CopyArgs a;
  std::memset(&a, 0, sizeof(a));
  a.k_pool = cache->k_pool;
  a.v_pool = cache->v_pool;
  a.page_bytes = (int64_t)cache->n_kv_heads * cache->page_size * cache->head_dim * elem_bytes(cache);
  a.layer_bytes = cache->n_pages * a.page_bytes;
  a.n_pages = cache->n_pages;
  a.block_table = block_table;
  a.payload = const_cast<void*>(payload);
  a.first_page = first_token / cache->page_size;
  a.n_block_pages = n_pages;
  a.n_tokens = hdr->n_tokens;
  a.n_layers = cache->n_layers;
  a.row_bytes = cache->head_dim * (int)elem_bytes(cache);
  a.Hkv = cache->n_kv_heads;
  a.D = cache->head_dim;
  a.relocate = d != 0;
  a.pairing = hdr->rope_pairing;
  if (a.relocate) {
    // cos/sin of d * theta_i in fp64, rounded once to fp32
    for (int i = 0; i < cache->head_dim / 2; ++i) {
      const double theta = std::pow(hdr->rope_base, -2.0 * i / cache->head_dim);
      const double ang = (double)d * theta;
      a.cs[2 * i] = (float)std::cos(ang);
      a.cs[2 * i + 1] = (float)std::sin(ang);
    }
  }
  if (!fits_grid(kvg::copy_workgroups(a, cache->dtype), 256)) return KVG_E_SHAPE;
  return hip_status(kvg::launch_graft(a, cache->dtype, static_cast<hipStream_t>(stream)));
}

size_t kvg_prefill_workspace_bytes(const kvg_cache* cache, const kvg_seqs* seqs, int32_t n_layers,
                                   int32_t chunk_len) {
  if (check_cache(cache) != KVG_OK || seqs == nullptr || n_layers <= 0 || chunk_len <= 0 || seqs->batch <= 0)
    return 0;
  if (use_mfma(cache)) return mfma_ws(cache, seqs, n_layers, chunk_len);
  return valu_ws(cache, seqs, n_layers, chunk_len).total;
}

int kvg_prefill_attn(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope, int32_t layer0,
                     int32_t n_layers, int32_t chunk_len, const void* q_raw, const void* k_raw,
                     const void* v_raw, float scale, float* out, void* ws, size_t ws_bytes, void* stream) {
  const int st = check_attn(cache, seqs, rope, layer0, n_layers, chunk_len, q_raw, k_raw, v_raw, scale, out);
  if (st != KVG_OK) return st;
  if (use_mfma(cache))
    return attn_mfma(cache, seqs, rope, layer0, n_layers, chunk_len, q_raw, k_raw, v_raw, scale, out, ws,
                     ws_bytes, static_cast<hipStream_t>(stream));
  return attn_valu(cache, seqs, rope, layer0, n_layers, chunk_len, q_raw, k_raw, v_raw, scale, out, ws,
                   ws_bytes, static_cast<hipStream_t>(stream));
}

size_t kvg_decode_workspace_bytes(const kvg_cache* cache, const kvg_seqs* seqs, int32_t n_layers) {
  if (check_cache(cache) != KVG_OK || seqs == nullptr || n_layers <= 0 || seqs->batch <= 0) return 0;
  return decode_ws(cache, seqs, n_layers).total;
}

int kvg_decode_attn(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope, int32_t layer0,
                    int32_t n_layers, const void* q_raw, const void* k_raw, const void* v_raw, float scale,
                    float* out, void* ws, size_t ws_bytes, void* stream) {
  const int st = kvg::decode_attn_check(cache, seqs, rope, layer0, n_layers, q_raw, k_raw, v_raw, scale, out);
  if (st != KVG_OK) return st;
  return kvg::decode_attn_launch(cache, seqs, rope, layer0, n_layers, q_raw, k_raw, v_raw, scale, out, ws, ws_bytes,
                                 static_cast<hipStream_t>(stream));
}

}  // extern "C"

namespace kvg {

int decode_attn_check(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope, int32_t layer0,
                      int32_t n_layers, const void* q_raw, const void* k_raw, const void* v_raw, float scale,
                      float* out) {
  return check_attn(cache, seqs, rope, layer0, n_layers, 1, q_raw, k_raw, v_raw, scale, out);
}

size_t decode_attn_ws_bytes(const kvg_cache* cache, const kvg_seqs* seqs, int32_t n_layers) {
  return decode_ws(cache, seqs, n_layers).total;
}

int decode_attn_launch(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope, int32_t layer0,
                       int32_t n_layers, const void* q_raw, const void* k_raw, const void* v_raw, float scale,
                       float* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  const DecodeWs w = decode_ws(cache, seqs, n_layers);
  if (ws == nullptr || ws_bytes < w.total) return KVG_E_WORKSPACE;
  const int n_split = n_split_max(seqs, 1);
  const int n_grid = decode_grid_splits(cache, seqs, layer0, n_layers);
  const int64_t n_blocks = (int64_t)n_layers * seqs->batch * cache->n_kv_heads * n_grid;
  const int64_t n_rows = (int64_t)n_layers * seqs->batch * cache->n_q_heads;
  if (!fits_grid(n_blocks, 256) || !fits_grid(n_rows, 256) || !append_fits(seqs, 1)) return KVG_E_SHAPE;
  if (shared_splits(cache, seqs) > 0) {
    const int nw = kvg::prefill_mfma_waves(cache->head_dim);
    const int64_t sh_waves = ((int64_t)seqs->batch + 31) / 32 * (cache->n_q_heads / cache->n_kv_heads);
    const int64_t sh_wg = (int64_t)n_layers * cache->n_kv_heads * shared_splits(cache, seqs) * ((sh_waves + nw - 1) / nw);
    if (!fits_grid(sh_wg, 64 * nw)) return KVG_E_SHAPE;
  }
  char* base = static_cast<char*>(ws);
  kvg::DecodeArgs a;
  std::memset(&a, 0, sizeof(a));
  a.k_pool = cache->k_pool;
  a.v_pool = cache->v_pool;
  a.layer_elems = layer_elems(cache);
  a.n_pages = cache->n_pages;
  a.block_tables = seqs->block_tables;
  a.ctx_lens = seqs->ctx_lens;
  a.start_pos = seqs->start_pos;
  a.q_raw = q_raw;
  a.k_raw = k_raw;
  a.v_raw = v_raw;
  a.out = out;
  a.part_ml = reinterpret_cast<float*>(base);
  a.part_acc = reinterpret_cast<float*>(base + w.ml);
  a.scale_log2 = scale * 1.4426950408889634f;
  a.Hq = cache->n_q_heads;
  a.Hkv = cache->n_kv_heads;
  a.D = cache->head_dim;
  a.group = cache->n_q_heads / cache->n_kv_heads;
  a.layer0 = layer0;
  a.n_layers = n_layers;
  a.batch = seqs->batch;
  a.max_pages = seqs->max_pages;
  a.max_ctx_len = seqs->max_ctx_len;
  a.n_split_max = n_split;
  a.shared_order = seqs->shared_tokens > 0 && seqs->batch > 1;
  a.n_shared_split = shared_splits(cache, seqs);
  a.n_split_grid = n_grid;
  a.pairing = rope->pairing;
  for (int i = 0; i < cache->head_dim / 2; ++i) a.theta[i] = std::pow(rope->base, -2.0 * i / cache->head_dim);
  if (fill_windows(cache, layer0, n_layers, a.window) != KVG_OK) return KVG_E_SHAPE;
  const hipStream_t hs = stream;
  if (a.n_shared_split > 0) {
    // Shared splits: the new token appended and the queries rotated into the workspace, then
    // the splits every sequence shares, read once for the whole batch on MFMA.  The split
    // kernel below appends the same token again (the same bytes) and skips those splits.
    uint16_t* qws = reinterpret_cast<uint16_t*>(base + w.ml + w.acc);
    uint16_t* qws_lo = reinterpret_cast<uint16_t*>(base + w.ml + w.acc + w.q / 2);
    kvg::AppendArgs ap = append_args(cache, seqs, rope, layer0, n_layers, 1, k_raw, v_raw);
    ap.q_raw = q_raw;
    ap.q_out = qws;
    ap.q_out_lo = qws_lo;
    ap.q_out_bf16 = 1;
    int sa = hip_status(kvg::launch_append(ap, cache->dtype, hs));
    if (sa != KVG_OK) return sa;
    kvg::PrefillArgs p;
    std::memset(&p, 0, sizeof(p));
    p.k_pool = cache->k_pool;
    p.v_pool = cache->v_pool;
    p.layer_elems = a.layer_elems;
    p.n_pages = cache->n_pages;
    p.block_tables = seqs->block_tables;
    p.ctx_lens = seqs->ctx_lens;
    p.q = qws;
    p.q_lo = qws_lo;
    p.part_acc = a.part_acc;
    p.part_ml = a.part_ml;
    p.scale_log2 = a.scale_log2;
    p.Hq = a.Hq;
    p.Hkv = a.Hkv;
    p.D = a.D;
    p.group = a.group;
    p.layer0 = layer0;
    p.n_layers = n_layers;
    p.batch = seqs->batch;
    p.chunk = 1;
    p.max_pages = seqs->max_pages;
    p.max_ctx_len = seqs->max_ctx_len;
    const int waves = (seqs->batch + 31) / 32 * a.group;                 // 32 sequences of one head per wave
    const int nw = kvg::prefill_mfma_waves(cache->head_dim);
    p.n_qt = (waves + nw - 1) / nw;
    p.n_split_max = n_split;
    p.n_shared_split = a.n_shared_split;
    p.shared_keys = kSplit;
    std::memcpy(p.window, a.window, sizeof(p.window));
    sa = hip_status(kvg::launch_shared_splits(p, cache->dtype, hs));
    if (sa != KVG_OK) return sa;
  }
  return hip_status(kvg::launch_decode(a, cache->dtype, hs));
}

}  // namespace kvg
