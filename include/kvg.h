/*
 * kvg.h -- C ABI of libkvg.so: byte-exact KV-state grafting on AMD Instinct MI355X (gfx950).
 *
 * The method (arXiv 2607.14431, "Byte-Exact KV-State Grafting"): the KV state S of a
 * processed prefix is captured once as a persistent block (deposit) and later
 * installed into a fresh context (graft) as the prefix [0, N) at its own positions,
 * new queries being computed fresh on top at [N, N + q) (Sec. 3.2).  At its own
 * position the graft leaves the logits byte-identical to a fresh computation
 * (Eq. 1: SHA-256 of the logit bytes equal); relocating a block to another
 * absolute offset re-rotates its rotary-encoded keys and is not byte-exact
 * (Sec. 4.2).
 *
 * Conventions shared by every entry point
 *  - All pointers named *_dev, and every pointer inside kvg_cache / kvg_seqs, are
 *    device pointers unless stated.  The caller allocates and owns all memory
 *    (pools, tables, payloads, outputs, workspaces).  The library allocates no
 *    device memory and keeps no state between calls; calls are re-entrant.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Kernels are enqueued on
 *    it and the call returns after enqueueing; results are visible after the
 *    caller synchronises the stream.  Apart from kvg_artifact_seal and
 *    kvg_artifact_verify (which wait for their digest), no call synchronises, copies to
 *    the host or clears memory with a runtime memset, so their launches can be captured
 *    into a HIP graph on `stream` and replayed.
 *  - Every call validates its arguments on the host before launching anything and
 *    returns a kvg_status.  No exception crosses the ABI.  A launch failure returns
 *    KVG_E_HIP; device faults surface at the caller's synchronisation.
 *  - Logical token index t in [0, len) of a sequence addresses the cache through
 *    its block table: physical page block_table[t / page_size], row t % page_size.
 *    The absolute position used by the rotary embedding is start_pos + t.
 *  - Kernels never read or write outside the pool, table, payload, output or
 *    workspace extents the arguments describe: block-table entries outside
 *    [0, n_pages) and context lengths outside [0, max_ctx_len] are skipped (the
 *    affected outputs are then unspecified), never dereferenced.
 *  - Reduction orders depend only on logical token indices, never on physical
 *    page ids, batch size, chunking of other sequences or the device's CU count,
 *    so the fresh path and the graft path produce identical bytes.  One exception is
 *    opt-in: a nonzero kvg_seqs.shared_tokens lets the attention calls compute the shared
 *    pages once for the batch, and a sequence's bytes then depend on that value and on
 *    whether the batch takes that path (see kvg_seqs); two calls with the same batch and
 *    value still give the same bytes.
 */
#ifndef KVG_H
#define KVG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KVG_OK = 0,
  KVG_E_INVAL = -1,       /* NULL pointer or negative/zero size where one is required   */
  KVG_E_SHAPE = -2,       /* head geometry or layer range does not match / unsupported  */
  KVG_E_DTYPE = -3,       /* storage dtype unsupported or artifact dtype differs         */
  KVG_E_POSITION = -4,    /* graft target position differs from the block's own position */
  KVG_E_CAPACITY = -5,    /* block table too short for the tokens addressed              */
  KVG_E_ALIGN = -6,       /* block start not page aligned, or a buffer not 16-byte aligned  */
  KVG_E_CORRUPT = -7,     /* artifact header inconsistent, or payload differs from its digest */
  KVG_E_HIP = -8,         /* a HIP launch or runtime call failed                           */
  KVG_E_WORKSPACE = -9    /* workspace smaller than the size query returned               */
} kvg_status;

/* Storage dtype of a cache.  FP8_E4M3 is OCP FP8 E4M3 (1 sign, 4 exponent bits with bias
 * 7, 3 mantissa bits; largest finite 448, codes 0x7F / 0xFF NaN), the KV-cache
 * quantization the paper lists among the serving settings that shape a block (Sec. 4.4):
 * its raw q/k/v inputs are bf16, stored keys (after rotation) and values are rounded once
 * to nearest even and saturate at +-448, and attention reads them back exactly (every
 * E4M3 value is a bf16 value).  A block's payload keeps the cache's bytes, so an fp8 block
 * is half the size of a bf16 one and its graft is the same byte copy. */
typedef enum { KVG_F32 = 0, KVG_BF16 = 1, KVG_FP8_E4M3 = 2 } kvg_dtype;

/* Rotary pairing of the D components: HALF pairs i with i + D/2, INTERLEAVED pairs
 * 2i with 2i + 1.  theta_i = base^(-2i/D), i in [0, D/2). */
typedef enum { KVG_ROPE_HALF = 0, KVG_ROPE_INTERLEAVED = 1 } kvg_rope_pairing;

typedef struct {
  double base;          /* e.g. 10000.0 */
  int32_t pairing;      /* kvg_rope_pairing */
  int32_t reserved;     /* must be 0 */
} kvg_rope;

/* Paged KV cache.  k_pool and v_pool each hold
 *   [n_layers][n_pages][n_kv_heads][page_size][head_dim]  elements of `dtype`,
 * keys stored after rotation at their absolute positions.
 * Supported: dtype F32, BF16 or FP8_E4M3; head_dim 64, 128 or 256; page_size 16;
 * n_q_heads a multiple of n_kv_heads with group n_q_heads / n_kv_heads in {1,2,4,8}.
 * Query head h reads KV head h / group (contiguous groups).
 * layer_window: NULL (every layer full causal) or a host array of n_layers windows: 0 =
 * full causal, W > 0 = a sliding-window layer whose row i attends keys i - W < j <= i
 * (the paper's model interleaves windowed and global layers and keeps full-size KV for the
 * windowed ones, Sec. 4.3; deposit and graft move every layer alike).  Attention calls copy
 * the windows of their layers into the launch; windows are supported for calls of at most
 * KVG_MAX_WINDOW_LAYERS layers. */
#define KVG_MAX_WINDOW_LAYERS 128

typedef struct {
  int32_t n_layers;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t page_size;
  int32_t dtype;        /* kvg_dtype */
  int64_t n_pages;      /* physical pages per layer */
  void* k_pool;
  void* v_pool;
  const int32_t* layer_window;   /* host [n_layers] or NULL */
} kvg_cache;

/* A batch of sequences for attention calls.  Metadata is read, never written.
 * shared_tokens (0 <= shared_tokens <= max_pages * page_size): 0, or a promise that
 * block_tables[b][i] is the same for every sequence b and every i < shared_tokens /
 * page_size (a window of pages the sequences share), and that every ctx_lens[b] >=
 * shared_tokens (no sequence appends into them).  kvg_decode_attn then orders its work
 * so that the sequences reading a shared page run together and, for bf16 and fp8 caches with
 * at most 4 query heads per KV head and a batch of two or more, computes the 512-key splits
 * inside the shared pages of full-attention layers once for the whole batch on MFMA (every
 * sequence's query against each shared page, read once), combining them with the
 * sequence's own splits as usual.  kvg_prefill_attn, under the same conditions and for a
 * chunk shorter than its row tile (32 x 8 / group rows per query head below head_dim 256,
 * 32 x 4 / group at 256), computes the attention of every sequence's chunk rows over the
 * shared pages' whole 512-key splits
 * once for the whole batch (each shared page read once per KV head and group of rows), the
 * rest per sequence, and combines the two partials of each row on full-attention layers;
 * its workspace then also holds those partials.  The results then depend on the value
 * (another summation order; within the same tolerance of the exact attention), and are
 * deterministic for a given value.  Other calls ignore it.  A broken promise gives
 * unspecified values, never an access outside the cache or the workspace. */
typedef struct {
  int32_t batch;
  int32_t max_pages;            /* entries per block-table row                       */
  int32_t max_ctx_len;          /* host-side upper bound of every ctx_lens[b]        */
  int32_t shared_tokens;        /* leading tokens shared by every sequence, see below */
  const int32_t* block_tables;  /* device [batch][max_pages] physical page ids        */
  const int32_t* ctx_lens;      /* device [batch] tokens already cached before the call */
  const int64_t* start_pos;     /* device [batch] absolute position of logical token 0 */
} kvg_seqs;

#define KVG_ARTIFACT_MAGIC 0x4147564Bu  /* "KVGA" little endian */
#define KVG_ARTIFACT_VERSION 2u

/* Host-side header describing a deposited block (96 bytes, no padding; header and payload
 * written one after the other are the block's file form).  The payload it describes is
 *   [n_layers][2 (K, V)][ceil(n_tokens / page_size)][n_kv_heads][page_size][head_dim]
 * elements of `dtype` in logical page order; rows at or beyond n_tokens in the last
 * page are zero.
 * digest: the payload's content digest (block digests, Sec. 4.11), filled by
 * kvg_artifact_seal: the payload is cut into leaves of digest_leaf_bytes bytes (one
 * page of one KV head, page_size * head_dim elements: the layout's natural unit), each
 * leaf hashed with SHA-256 (FIPS 180-4), and the leaf digests reduced level by level to a
 * Merkle root (nodes 2i and 2i+1 combine into SHA-256(0x01 || left || right), an odd last
 * node moves up unchanged).  digest_leaf_bytes == 0: not sealed. */
typedef struct {
  uint32_t magic;
  uint32_t version;
  int32_t dtype;
  int32_t n_layers;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t page_size;
  int32_t n_tokens;
  int64_t own_pos;      /* absolute position of the block's first token at capture */
  double rope_base;
  int32_t rope_pairing;
  uint32_t digest_leaf_bytes;
  uint64_t payload_bytes;
  uint8_t digest[32];
} kvg_artifact_hdr;

/* Library identity string (backend, version, target), e.g. "kvg 0.1 gfx950". */
const char* kvg_version(void);

/* Human-readable name of a kvg_status value. */
const char* kvg_status_str(int status);

/* Bytes of the payload of an n_tokens block for this cache geometry; 0 on bad args. */
size_t kvg_payload_bytes(const kvg_cache* cache, int32_t n_tokens);

/* Fill a header for an n_tokens block captured at own_pos (not sealed: digest zeroed,
 * digest_leaf_bytes 0).  Errors: KVG_E_INVAL, KVG_E_SHAPE, KVG_E_DTYPE. */
int kvg_artifact_header_init(const kvg_cache* cache, int32_t n_tokens, int64_t own_pos,
                             const kvg_rope* rope, kvg_artifact_hdr* hdr_out);

/* KV-append: the fresh computation of new tokens' keys and values (Sec. 3.2, new
 * queries computed fresh on top).  For each sequence b and i in [0, chunk_len), the
 * token at logical index ctx_lens[b] + i and position start_pos[b] + ctx_lens[b] + i:
 *   K <- round(R(pos) k_raw)   (rotation in fp32 from fp64-derived cos/sin, rounded
 *                               to nearest even in the storage dtype)
 *   V <- v_raw
 * written through the block table.  Layers [layer0, layer0 + n_layers) of the cache.
 * k_raw_dev, v_raw_dev: [n_layers][batch][chunk_len][n_kv_heads][head_dim] of the
 * cache dtype (bf16 for an fp8 cache, whose values are rounded to fp8 when stored).
 * Errors: KVG_E_INVAL, KVG_E_SHAPE, KVG_E_CAPACITY (max_ctx_len + chunk_len >
 * max_pages * page_size), KVG_E_HIP. */
int kvg_append(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope,
               int32_t layer0, int32_t n_layers, int32_t chunk_len,
               const void* k_raw_dev, const void* v_raw_dev, void* stream);

/* Deposit (state capture, Sec. 3.1-3.2): gather tokens [first_token, first_token +
 * n_tokens) of one sequence, all layers, K and V, into payload_dev (layout above,
 * kvg_payload_bytes(cache, n_tokens) bytes, zero tail).  A pure byte move.
 * block_table_dev: that sequence's row, table_len entries.
 * Errors: KVG_E_INVAL, KVG_E_ALIGN (first_token % page_size), KVG_E_CAPACITY
 * (table shorter than the block's pages), KVG_E_HIP. */
int kvg_deposit(const kvg_cache* cache, const int32_t* block_table_dev, int32_t table_len,
                int32_t first_token, int32_t n_tokens, void* payload_dev, void* stream);

/* Workspace bytes kvg_artifact_seal and kvg_artifact_verify need for this header's payload
 * (0 if the header's geometry is invalid). */
size_t kvg_artifact_digest_workspace_bytes(const kvg_artifact_hdr* hdr);

/* Seal a deposited block (block digests, Sec. 4.11; the paper identifies stored blocks by
 * SHA-256 and verifies restores by byte equality, Eq. 1): compute the digest defined at
 * kvg_artifact_hdr of payload (device memory, or host-pinned memory the device can read;
 * 16-byte aligned) on the device, then write hdr->digest and hdr->digest_leaf_bytes.
 * Blocks: the call enqueues on `stream` and waits for it (the host needs the value).
 * ws_dev: kvg_artifact_digest_workspace_bytes() bytes of device scratch.
 * Errors: KVG_E_INVAL, KVG_E_CORRUPT (magic, version, or payload_bytes inconsistent with
 * the header's geometry), KVG_E_ALIGN, KVG_E_WORKSPACE, KVG_E_HIP. */
int kvg_artifact_seal(kvg_artifact_hdr* hdr, const void* payload, void* ws_dev, size_t ws_bytes, void* stream);

/* Verify a block before grafting it, e.g. one read back from a file in another process
 * (cross-context restore, Sec. 3.2): recompute the payload's digest as kvg_artifact_seal
 * does and compare it with hdr->digest.  Blocks like kvg_artifact_seal.
 * Returns KVG_OK when they are equal, KVG_E_CORRUPT when they differ, when the header is not
 * sealed or when its fields are inconsistent; other errors as kvg_artifact_seal. */
int kvg_artifact_verify(const kvg_artifact_hdr* hdr, const void* payload, void* ws_dev, size_t ws_bytes,
                        void* stream);

#define KVG_GRAFT_ALLOW_RELOCATE 1

/* Graft (state restore, Sec. 3.2; relocation, Sec. 4.2): scatter the payload's valid
 * rows into the pages named by block_table_dev, starting at logical token first_token
 * (page aligned).  Rows past the block in its last page are left untouched.
 * target_pos is the absolute position the block's first token will have; with
 * d = target_pos - hdr->own_pos:
 *   d == 0: a byte move (the restored pages equal the payload bit for bit);
 *   d != 0: requires KVG_GRAFT_ALLOW_RELOCATE; keys are re-rotated by d (fp32
 *           rotation with cos/sin of d * theta_i computed in fp64 on the host,
 *           rounded to the storage dtype), values copied.  Not byte-exact against a
 *           fresh computation at the new offset (Sec. 4.2).
 * payload: device memory or host-pinned memory the device can read.  The graft is a plain
 * asynchronous copy: it does not read the digest (kvg_artifact_verify checks the payload
 * against it first).
 * Errors: KVG_E_INVAL, KVG_E_CORRUPT (magic/version/payload_bytes), KVG_E_SHAPE /
 * KVG_E_DTYPE (header geometry differs from the cache), KVG_E_POSITION,
 * KVG_E_ALIGN, KVG_E_CAPACITY, KVG_E_HIP. */
int kvg_graft(const kvg_cache* cache, const kvg_artifact_hdr* hdr, const void* payload,
              const int32_t* block_table_dev, int32_t table_len, int32_t first_token,
              int64_t target_pos, int32_t flags, void* stream);

/* Workspace bytes kvg_prefill_attn needs for this batch (0 on bad args). */
size_t kvg_prefill_workspace_bytes(const kvg_cache* cache, const kvg_seqs* seqs,
                                   int32_t n_layers, int32_t chunk_len);

/* Chunked-prefill attention for a suffix on top of the cached (e.g. grafted) prefix
 * (Sec. 3.2; the cache-hit prefill after a restore, Sec. 4.4).  First appends the
 * chunk's K/V exactly as kvg_append, then for every new row i of sequence b (logical
 * index n = ctx_lens[b] + i) computes, per query head h,
 *   out = softmax_j( (R(pos_n) q_h . K_{h/group, j}) * scale ) V_{h/group, j},  j <= n
 * with fp32 softmax and accumulation (j > n - W as well in a layer with window W).
 * bf16 and fp8 caches with at most 4 query heads per KV head use bf16 MFMA for Q K^T and
 * P V (each rotated query carried as a bf16 high part and a bf16 low part, both multiplied
 * with every key, so a score is as accurate as with the fp32 query; P rounded to bf16; fp8
 * rows widened to bf16 exactly); fp32 caches, and 8 query heads per KV head, use fp32
 * vector arithmetic (bf16 and fp8 caches there: the same query parts, P rounded to bf16).
 * q_raw_dev: [n_layers][batch][chunk_len][n_q_heads][head_dim] of the raw dtype (the cache
 * dtype, bf16 for an fp8 cache), pre-rotation;
 * k_raw_dev, v_raw_dev as kvg_append; out_dev: [n_layers][batch][chunk_len][n_q_heads]
 * [head_dim] fp32.  ws_dev: kvg_prefill_workspace_bytes() bytes (scratch, contents
 * undefined after the call).
 * Errors: as kvg_append, plus KVG_E_WORKSPACE, and KVG_E_SHAPE / KVG_E_INVAL for
 * windows on more than KVG_MAX_WINDOW_LAYERS layers / a negative window. */
int kvg_prefill_attn(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope,
                     int32_t layer0, int32_t n_layers, int32_t chunk_len,
                     const void* q_raw_dev, const void* k_raw_dev, const void* v_raw_dev,
                     float scale, float* out_dev, void* ws_dev, size_t ws_bytes, void* stream);

/* Workspace bytes kvg_decode_attn needs (0 on bad args). */
size_t kvg_decode_workspace_bytes(const kvg_cache* cache, const kvg_seqs* seqs, int32_t n_layers);

/* Decode attention over the restored context (Sec. 4.3 "advancing by a single
 * token"; Sec. 4.4 decode after restore): one new token per sequence, appended as
 * kvg_append with chunk_len = 1, then attended inclusively over keys [0, ctx_lens[b]]
 * (the last W of them in a layer with window W; ranges entirely before the window are
 * skipped).
 * Grouped-query split-K over fixed 512-token ranges of logical index: each range yields a
 * partial (reference max, sum, weighted V) in fp32 and the partials are combined in
 * ascending range order, so the bytes depend neither on the batch nor on which path filled
 * the cache.  bf16 and fp8 caches hold the rotated query as a bf16 high and low part (each
 * score the sum of both products) and round the softmax weights to bf16 (as the MFMA prefill
 * rounds P), the sum of weights taking the rounded values; fp32 caches keep fp32 queries and
 * weights.  Two
 * launches: the split kernel (which also rotates the queries and appends the new token)
 * and the combine kernel.  Layouts as kvg_prefill_attn with chunk_len = 1.
 * ws_dev: kvg_decode_workspace_bytes() bytes of scratch (contents undefined after the call).
 * Errors: as kvg_prefill_attn. */
int kvg_decode_attn(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope,
                    int32_t layer0, int32_t n_layers,
                    const void* q_raw_dev, const void* k_raw_dev, const void* v_raw_dev,
                    float scale, float* out_dev, void* ws_dev, size_t ws_bytes, void* stream);

/* Decode on the library's own workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same computation as kvg_decode_attn (same kernels, same bytes), with the workspace taken
 * from a fixed device array of KVG_NOALLOC_SCRATCH_BYTES bytes that the library holds on every
 * device it runs on until the process ends (its address is looked up once per device, on the
 * first call there).  The call itself allocates nothing.  Calls whose workspace
 * (kvg_decode_workspace_bytes) exceeds the array return KVG_E_WORKSPACE before launching
 * anything.  All calls on one device share the array and keep no state in it between calls:
 * calls that overlap on one device (several streams or threads) race and must be serialised
 * by the caller.  Errors: as kvg_decode_attn, and KVG_E_HIP when the array's address cannot
 * be taken. */
#define KVG_NOALLOC_SCRATCH_BYTES (256u << 20)
int kvg_decode_attn_noalloc(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope,
                            int32_t layer0, int32_t n_layers,
                            const void* q_raw_dev, const void* k_raw_dev, const void* v_raw_dev,
                            float scale, float* out_dev, void* stream);

/* ---- Content digests of an artifact (block digests, Sec. 4.11; the paper's deposit-side
 * hashing is closed, Sec. 3.1).  These calls work on any device buffer, typically a
 * deposited payload.  SHA-256 is FIPS 180-4.  All three launch on `stream`, clear their
 * own workspace with kernels (no memset), keep no state between calls and are
 * deterministic. */

/* Leaf digests: the buffer [0, n_bytes) cut into consecutive leaves of leaf_bytes (a
 * positive multiple of 64; the last leaf holds the remainder), and the SHA-256 of each
 * leaf written to digests_dev[32 i .. 32 i + 31] (device, 32 * ceil(n_bytes / leaf_bytes)
 * bytes).  One lane hashes one leaf, so small leaves (a page slab, 8 KiB at the 12B-class
 * shapes) keep the device busy.  data_dev must be 16-byte aligned.
 * Errors: KVG_E_INVAL (null pointer, n_bytes == 0, bad leaf_bytes), KVG_E_ALIGN,
 * KVG_E_HIP. */
int kvg_leaf_digests(const void* data_dev, uint64_t n_bytes, uint32_t leaf_bytes,
                     uint8_t* digests_dev, void* stream);

/* Workspace bytes kvg_merkle_root needs for n_leaves leaves (0 if n_leaves == 0). */
size_t kvg_merkle_workspace_bytes(uint64_t n_leaves);

/* Merkle root of n_leaves 32-byte digests (device), level by level: nodes 2i and 2i+1 of
 * a level combine into SHA-256(0x01 || left || right), an odd last node moves up
 * unchanged, the root of a single leaf is that leaf's digest.  root_dev: 32 bytes of
 * device memory.  ws_dev: kvg_merkle_workspace_bytes(n_leaves) bytes of scratch.
 * Errors: KVG_E_INVAL, KVG_E_WORKSPACE, KVG_E_HIP. */
int kvg_merkle_root(const uint8_t* digests_dev, uint64_t n_leaves, uint8_t* root_dev,
                    void* ws_dev, size_t ws_bytes, void* stream);

/* Workspace bytes kvg_dedup_map needs for n_leaves leaves (0 if n_leaves == 0). */
size_t kvg_dedup_workspace_bytes(uint64_t n_leaves);

/* Content-addressed dedup map: first_index_dev[i] = the smallest j with digest j equal to
 * digest i (int64, device, n_leaves entries).  Leaves are matched through an open-
 * addressing table keyed by the first 8 digest bytes and every match is confirmed on all
 * 32 bytes; a leaf whose key collides with a different digest is left unresolved
 * (first_index -1) and counted in *n_unresolved_dev (int32, device).
 * ws_dev: kvg_dedup_workspace_bytes(n_leaves) bytes of scratch.
 * Errors: KVG_E_INVAL, KVG_E_WORKSPACE, KVG_E_HIP. */
int kvg_dedup_map(const uint8_t* digests_dev, uint64_t n_leaves, int64_t* first_index_dev,
                  int32_t* n_unresolved_dev, void* ws_dev, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------
 * Logits (Eq. 1-2; soft cap, Sec. 4.2).  The verdict on a graft is taken on the logits at a
 * position: their bytes (SHA-256 equality; kvg_leaf_digests with leaf_bytes = 4 * vocab
 * hashes each row), the KL divergence of the two softmax distributions and their argmax.
 * A synthetic head stands in for the model's: the caller supplies hidden vectors (e.g. the
 * last layer's attention outputs, heads concatenated) and a bf16 weight matrix. */

/* Bytes of the packed head weights for a [vocab][hidden] matrix (0 for a non-positive size). */
size_t kvg_logits_packed_bytes(int32_t vocab, int32_t hidden);

/* Packs the head weights once (as a model loader would): w_dev, bf16 bits [vocab][hidden]
 * row-major, into packed_dev (kvg_logits_packed_bytes bytes), a layout of the library's
 * own in which every MFMA operand fragment is 1 KiB of consecutive bytes and each block of 32
 * vocabulary rows is one contiguous run (rows past vocab are zero).  Both device, 16-byte
 * aligned.  Errors: KVG_E_INVAL, KVG_E_SHAPE (hidden not a multiple of 128), KVG_E_ALIGN,
 * KVG_E_HIP. */
int kvg_logits_pack(const uint16_t* w_dev, int32_t vocab, int32_t hidden, uint16_t* packed_dev, void* stream);

/* Workspace bytes kvg_logits needs (0 for a non-positive size). */
size_t kvg_logits_workspace_bytes(int32_t rows, int32_t hidden);

/* logits[r][v] = cap * tanh(z / cap) with z = sum_k bf16(hidden[r][k]) * w[v][k], or z when
 * cap == 0.  hidden_dev: fp32 [rows][hidden], rounded to bf16 (nearest even) before the
 * product; w_packed_dev: the weights as kvg_logits_pack left them; logits_dev: fp32
 * [rows][vocab]; all device, 16-byte aligned.  The products accumulate in fp32 on MFMA in an
 * order fixed by the shapes alone, so equal inputs give equal bytes.  Up to 128 rows read the
 * weights once (up to 32 at the full rate); every further 128 rows read them again.  ws_dev:
 * kvg_logits_workspace_bytes(rows, hidden) bytes of scratch.
 * Errors: KVG_E_INVAL (null pointer, non-positive size, cap negative or not finite),
 * KVG_E_SHAPE (hidden not a multiple of 128, sizes too large), KVG_E_ALIGN,
 * KVG_E_WORKSPACE, KVG_E_HIP. */
int kvg_logits(const float* hidden_dev, int32_t rows, int32_t hidden, const uint16_t* w_packed_dev, int32_t vocab,
               float cap, float* logits_dev, void* ws_dev, size_t ws_bytes, void* stream);

/* Per row r of two logit sets a, b (fp32 [rows][vocab], device): kl_dev[r] =
 * KL(softmax(a_r) || softmax(b_r)) in fp64 (fixed-order sums: byte-equal rows give exactly
 * 0), argmax_a_dev[r] / argmax_b_dev[r] = the first index of each row's maximum (int32).
 * All outputs device.  Errors: KVG_E_INVAL, KVG_E_HIP. */
int kvg_logit_compare(const float* a_dev, const float* b_dev, int32_t rows, int32_t vocab, double* kl_dev,
                      int32_t* argmax_a_dev, int32_t* argmax_b_dev, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVG_H */
