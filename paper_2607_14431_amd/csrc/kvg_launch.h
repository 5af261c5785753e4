// Host-side launchers of the libkvg kernels (implemented next to each kernel).
#pragma once

#include <hip/hip_runtime.h>

#include "kvg_device.h"

namespace kvg {

hipError_t launch_append(const AppendArgs& a, int bf16, hipStream_t stream);
hipError_t launch_deposit(const CopyArgs& a, hipStream_t stream);
hipError_t launch_graft(const CopyArgs& a, int bf16, hipStream_t stream);
hipError_t launch_attn_valu(const AttnArgs& a, int bf16, hipStream_t stream);
hipError_t launch_prefill_mfma(const PrefillArgs& a, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs& a, int bf16, hipStream_t stream);

}  // namespace kvg
