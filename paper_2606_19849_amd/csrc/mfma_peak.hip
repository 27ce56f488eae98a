// Sustained bf16 matrix-core throughput (measurement helper, libvico_bench.so).
//
// Register-only MFMA chains: no memory traffic inside the loop, so the rate is
// set by the matrix cores and the engine clock the chip holds under that load.

#include <hip/hip_runtime.h>

#include "vico_bench.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 512;
constexpr int kLdsBytes = 80 * 1024;   // dynamic LDS per work-group, more than half of the CU's 160 KiB: one work-group per CU

__global__ __launch_bounds__(kThreads) void mfma_peak_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (lane + e));
    b[e] = (__bf16)(0.002f * (lane - e));
  }
  f32x16 c0{}, c1{}, c2{}, c3{};
  c1[0] = 1.f; c2[0] = 2.f; c3[0] = 3.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, a, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, a, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, b, c3, 0, 0, 0);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 16; ++e) s += c0[e] + c1[e] + c2[e] + c3[e];
  if (lane == 0) sink[blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)] = s;
}

}  // namespace

extern "C" int32_t vico_bench_mfma_peak(int32_t work_groups, int32_t iters, float* sink, void* stream) {
  if (work_groups < 1 || iters < 1 || sink == nullptr) return VICO_ERR_INVALID_ARG;
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute((const void*)mfma_peak_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes) !=
        hipSuccess)
      return VICO_ERR_HIP;
    attr_set = true;
  }
  hipLaunchKernelGGL(mfma_peak_kernel, dim3(work_groups), dim3(kThreads), kLdsBytes, (hipStream_t)stream, iters, sink);
  return hipGetLastError() == hipSuccess ? VICO_OK : VICO_ERR_HIP;
}
