// Host-side launchers of the libkvg kernels (implemented next to each kernel).
#pragma once

#include <hip/hip_runtime.h>

#include "kvg_device.h"

namespace kvg {

// `dtype` is the cache's storage dtype code (kDtypeF32, kDtypeBf16, kDtypeFp8).
hipError_t launch_append(const AppendArgs& a, int dtype, hipStream_t stream);
hipError_t launch_deposit(const CopyArgs& a, hipStream_t stream);
hipError_t launch_graft(const CopyArgs& a, int dtype, hipStream_t stream);
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

}  // namespace kvg
