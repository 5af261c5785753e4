// Host-side launchers of the libkvg kernels (implemented next to each kernel).
#pragma once

#include <hip/hip_runtime.h>

#include "kvg.h"
#include "kvg_device.h"

namespace kvg {

// `dtype` is the cache's storage dtype code (kDtypeF32, kDtypeBf16, kDtypeFp8).
hipError_t launch_append(const AppendArgs& a, int dtype, hipStream_t stream);
hipError_t launch_deposit(const CopyArgs& a, hipStream_t stream);
hipError_t launch_graft(const CopyArgs& a, int dtype, hipStream_t stream);
// workgroups (256 threads each) of the deposit's and of the graft's launch (own position or
// relocated), for the host's launch-size checks
int64_t copy_workgroups(const CopyArgs& a, int dtype);
hipError_t launch_attn_valu(const AttnArgs& a, int dtype, hipStream_t stream);
hipError_t launch_prefill_mfma(const PrefillArgs& a, int dtype, hipStream_t stream);
// waves (32 query rows each) per workgroup of the MFMA prefill at head_dim D; a workgroup
// covers 32 * waves / group rows of each of the group's query heads
int prefill_mfma_waves(int D);
// decode partials of splits [0, a.n_shared_split) of every full-attention layer, for a batch
// whose sequences share those pages; a.q holds the rotated queries [n_layers][batch][Hq][D]
hipError_t launch_shared_splits(const PrefillArgs& a, int dtype, hipStream_t stream);
// a suffix prefill over shared pages: out = the rows' n_split_max partials combined in order
hipError_t launch_prefill_combine(const PrefillArgs& a, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs& a, int dtype, hipStream_t stream);


// The decode call split at its workspace (kvg_api.cpp): argument validation, the workspace
// size, and the launches on a given workspace (which is checked against the size).
int decode_attn_check(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope, int32_t layer0,
                      int32_t n_layers, const void* q_raw, const void* k_raw, const void* v_raw, float scale,
                      float* out);
size_t decode_attn_ws_bytes(const kvg_cache* cache, const kvg_seqs* seqs, int32_t n_layers);
int decode_attn_launch(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope, int32_t layer0,
                       int32_t n_layers, const void* q_raw, const void* k_raw, const void* v_raw, float scale,
                       float* out, void* ws, size_t ws_bytes, hipStream_t stream);

}  // namespace kvg
