// vico_gather_attn_noalloc: vico_gather_attn with the key-range partials in a
// fixed device array owned by the library, for callers that cannot allocate
// (code under HIP graph capture, tight serving loops).  It launches the same
// kernels as vico_gather_attn; only where the partials live differs.

#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <stdint.h>

#include "vico.h"
#include "vico_internal.h"

namespace {

constexpr int64_t kScratchBytes = VICO_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

}  // namespace

// One copy per GPU the library runs on, held until the process ends.  In
// host code this name is not a device address: the kernels only ever see the
// address hipGetSymbolAddress reports for the current device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

std::mutex g_mu;
std::atomic<void*> g_scratch[kMaxDevices];

// Workspace source of vico_gather_attn_noalloc: the current device's copy of
// `scratch`, whose address is looked up once per device (the first call made
// with that device current).  A request beyond the array fails before any
// HIP call.
int scratch_workspace(int64_t need, void** ws, int64_t* ws_bytes) {
  if (need > kScratchBytes) return VICO_ERR_SCRATCH;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return vico::record_hip_failure(e);
  if (dev < 0 || dev >= kMaxDevices) return VICO_ERR_UNSUPPORTED;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p) return vico::record_hip_failure(e != hipSuccess ? e : hipErrorInvalidSymbol);
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *ws = p;
  *ws_bytes = kScratchBytes;
  return VICO_OK;
}

}  // namespace

extern "C" {

int vico_gather_attn_noalloc(const void* q, int32_t q_len, const void* tail_k, const void* tail_v, int32_t tail_len,
                             const void* sink_k, const void* sink_v, int32_t sink_len, const void* store_k,
                             const void* store_v, int32_t store_slots, const int64_t* seg_start,
                             const int32_t* seg_len, int32_t num_segments, int64_t keys_hint, int32_t num_q_heads,
                             int32_t num_kv_heads, int32_t head_dim, float softmax_scale, void* out,
                             int32_t out_dtype, float* lse_out, int32_t num_splits, void* stream) {
  // Every partial the merge reads is written earlier in the same call, so
  // the array needs no clearing between calls.
  return vico::gather_attn_entry(q, q_len, tail_k, tail_v, tail_len, sink_k, sink_v, sink_len, store_k, store_v,
                                 store_slots, seg_start, seg_len, num_segments, keys_hint, num_q_heads,
                                 num_kv_heads, head_dim, softmax_scale, out, out_dtype, lse_out, num_splits,
                                 nullptr, 0, stream, &scratch_workspace);
}

}  // extern "C"
