// Measurement helper for the roofline figures of libvico.
//
// Not part of the attention path: it lives in its own library,
// libvico_bench.so, which the benchmark loads to put the chunk kernel's MFMA
// rate next to the rate the matrix cores sustain on the same GPU in the same
// process (the published dense peak assumes the 2.4 GHz peak engine clock,
// which the chip does not hold while every CU keeps its matrix cores busy).
#ifndef VICO_BENCH_H_
#define VICO_BENCH_H_

#include <stdint.h>

#include "vico.h"

#ifdef __cplusplus
extern "C" {
#endif

// Sustained bf16 matrix-core throughput.
//   Launches `work_groups` work-groups of 512 threads (8 waves) on `stream`
//   (asynchronous).  Each work-group holds 80 KiB of LDS so that one runs per
//   CU, i.e. two waves per SIMD as in the chunk attention kernel.  Each wave
//   issues `iters` x 32 v_mfma_f32_32x32x16_bf16 on register operands in four
//   independent accumulation chains and writes one float per wave to `sink`
//   (device memory, work_groups * 8 floats, caller-owned) so that the work is
//   kept.  Flops per call: work_groups * 8 * iters * 32 * 32768.
//   Returns VICO_OK; VICO_ERR_INVALID_ARG if work_groups < 1, iters < 1 or
//   sink is NULL; VICO_ERR_HIP if the launch fails.
int32_t vico_bench_mfma_peak(int32_t work_groups, int32_t iters, float* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif  // VICO_BENCH_H_
