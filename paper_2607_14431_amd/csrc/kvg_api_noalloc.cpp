// kvg_decode_attn_noalloc: the decode call on a workspace the library holds itself, for callers
// that cannot allocate (declaration and contract in include/kvg.h).
//
// The workspace is a file-scope device array of fixed size; each device the library runs on
// holds its own copy until the process ends.  On the first call on a device its address is
// taken once with hipGetSymbolAddress (with that device current) and kept per device: in host
// code the array's name is only a stand-in, so kernels always receive that address.  Every
// call on a device shares its array: calls that overlap on one device (other streams, other
// threads) race.  The decode kernels write every partial they read back within a call, so
// nothing has to be cleared between calls.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kvg.h"
#include "kvg_launch.h"

namespace {

constexpr size_t kScratchBytes = size_t(KVG_NOALLOC_SCRATCH_BYTES);
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];      // per device: the array's device address, once taken

// The current device's scratch address; taken on the first call on that device.
int device_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return KVG_E_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return KVG_E_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return KVG_OK;
}

}  // namespace

extern "C" {

int kvg_decode_attn_noalloc(const kvg_cache* cache, const kvg_seqs* seqs, const kvg_rope* rope, int32_t layer0,
                            int32_t n_layers, const void* q_raw, const void* k_raw, const void* v_raw, float scale,
                            float* out, void* stream) {
  int st = kvg::decode_attn_check(cache, seqs, rope, layer0, n_layers, q_raw, k_raw, v_raw, scale, out);
  if (st != KVG_OK) return st;
  const size_t need = kvg::decode_attn_ws_bytes(cache, seqs, n_layers);
  if (need > kScratchBytes) return KVG_E_WORKSPACE;
  void* ws = nullptr;
  if ((st = device_scratch(&ws)) != KVG_OK) return st;
  return kvg::decode_attn_launch(cache, seqs, rope, layer0, n_layers, q_raw, k_raw, v_raw, scale, out, ws,
                                 kScratchBytes, static_cast<hipStream_t>(stream));
}

}  // extern "C"
