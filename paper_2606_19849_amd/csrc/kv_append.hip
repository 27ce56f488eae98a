// Ring-buffer append of a chunk's K/V into the bounded visual cache.
//
// ring[(H + j) mod R] <- chunk[j] for every token j of the chunk, for K and V
// (the cache that bounds what later chunks see; ViCoStream Sec. 3, "LLM
// Prefilling and Decoding").  Token rows are contiguous, so the destination
// is at most two contiguous runs of slots; each thread moves one 16-byte
// unit with one load and one store, consecutive threads consecutive units:
// fully coalesced on both sides.  The wrap is one compare-and-subtract.  (The
// split merge performs the same copy with append_units when an attention call
// appends its chunk.)

#include "vico_internal.h"

namespace vico {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// blockIdx.y picks K (0) or V (1), so source and destination stay scalar
__global__ __launch_bounds__(256) void kv_append_kernel(AppendArgs a) {
  const int upt = a.row_elems >> 3;                  // 16-byte units per token row
  const int64_t total = (int64_t)a.C * upt;
  const uint16_t* src = blockIdx.y ? a.vc : a.kc;
  uint16_t* dst = blockIdx.y ? a.rv : a.rk;
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < total; u += step) {
    const int j = (int)(u / upt);
    const int c = (int)(u - (int64_t)j * upt);
    int slot = a.p0 + j;
    if (slot >= a.R) slot -= a.R;
    *(u32x4*)(dst + (int64_t)slot * a.row_elems + c * 8) = *(const u32x4*)(src + (int64_t)j * a.row_elems + c * 8);
  }
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, hipStream_t stream) {
  const int64_t total = (int64_t)a.C * (a.row_elems >> 3);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)blocks, 2), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vico
