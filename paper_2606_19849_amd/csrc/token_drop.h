// Internal declarations of the temporal token dropping kernels (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vico {

// Temporal token dropping over B chunks of C frames of n_f tokens of dm features.
struct DropArgs {
  const uint16_t* frames;   // [B][C][n_f][dm] bf16
  const uint16_t* prev;     // [n_f][dm] frame before the batch (C == 1), may be null
  uint8_t* keep;            // [B][n_f] 1 = position kept
  float* sim;               // [B][n_f] smallest pairwise cosine, may be null
  uint16_t* out;            // [B*C*n_f][dm] retained tokens in stream order, may be null
  int32_t* out_index;       // [B*C*n_f] flat source row of each retained token
  int32_t* out_count;       // [1]
  void* ws;                 // single-pass control block (temporal_drop_workspace_bytes), null: two passes
  uint64_t epoch;           // single pass: this call's tag of the control words (nonzero, 52 bits)
  uint64_t wait_ticks;      // single pass: longest wait for another group, in 100 MHz ticks
  int B, C, n_f, dm;
  float tau;
};

hipError_t launch_temporal_drop(const DropArgs& a, hipStream_t stream);
// Workspace bytes of the single-pass drop, 0 where that schedule does not apply.
int64_t temporal_drop_workspace_bytes(int B, int C, int n_f, int dm);

}  // namespace vico
