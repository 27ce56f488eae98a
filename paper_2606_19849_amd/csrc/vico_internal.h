// Internal declarations shared by the HIP sources of libvico (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vico {

// Tile geometry of the attention kernel.  A work-group of 8 waves (two per
// SIMD) owns kBlockM = 256 query rows -- tokens of one query head, or packed
// (token, query head) pairs of the query heads of one KV head, token-major;
// each wave owns kRowBlocks = 1 block of 32 rows.  Keys are walked in tiles of kKeyTile,
// double-buffered in LDS (32 KiB per 64 keys at head_dim 128); one
// work-group per CU, so every K/V tile in LDS serves 256 rows.
constexpr int kThreads = 512;
constexpr int kRowBlocks = 1;
constexpr int kBlockM = (kThreads / 64) * kRowBlocks * 32;
constexpr int kKeyTile = 64;
constexpr int kBuffers = 2;
constexpr int kNumCUs = 256;        // MI355X: 8 XCDs x 32 CUs
constexpr int kWgPerCU = 1;
constexpr int kMaxSplits = 16;
constexpr int kAutoSplits = 16;     // most key splits the planner picks by itself (the row merge reads up to 16 parts at once)
constexpr int kMinSplitTiles = 8;   // fewest key tiles per split the planner picks by itself


// Everything the attention kernels need, resolved on the host.
struct AttnArgs {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const uint16_t* sink_k;
  const uint16_t* sink_v;
  const uint16_t* ring_k;
  const uint16_t* ring_v;
  void* out;
  float* lse;          // may be null
  float* ws_o;         // [splits][Hq][C][D] fp32, null when splits == 1
  float* ws_lse;       // [splits][Hq][C] fp32 (log2 units)
  int C, S, R, Wv, ws; // ws = first window slot = (H - Wv) mod R
  int Hq, Hkv, D;
  int splits;          // partial results per row merged at the end (1: none)
  int balanced;        // 1: work-groups take equal shares of all key tiles
  int pack;            // query heads packed into a row tile (divides Hq / Hkv): row r of a head
                       // group is token r / pack of query head (group base) + r % pack
  int64_t total_tiles; // balanced mode: key tiles summed over all row tiles and heads
  int out_f32;
  int bidir;           // 1: every chunk row sees the whole chunk (no causal mask)
  float scale_log2;    // softmax scale * log2(e)
  uint16_t* app_rk;    // append after attending (null: no append): ring K, V
  uint16_t* app_rv;
  int app_p0;          // first ring slot written = hist_len mod R
};

// Short-query attention over gathered key segments: query rows are the last
// Lq of T tail tokens; keys = sink ++ store segments ++ tail (causal).
constexpr int kGatherThreads = 512;  // 8 waves x 32 packed rows per work-group
constexpr int kMaxSegments = 2048;   // segment table entries per call
constexpr int kMaxGatherParts = 64;  // key-range parts per row tile
struct GatherArgs {
  const uint16_t* q;        // [Lq][Hq][D]
  const uint16_t* tail_k;   // [T][Hkv][D]
  const uint16_t* tail_v;
  const uint16_t* sink_k;   // [S][Hkv][D]
  const uint16_t* sink_v;
  const uint16_t* store_k;  // [cap][Hkv][D]
  const uint16_t* store_v;
  const int64_t* seg_start; // [n_segs] first store slot of each segment
  const int32_t* seg_len;   // [n_segs]
  void* out;                // [Lq][Hq][D]
  float* lse;               // [Hq][Lq], may be null
  float* ws_o;              // [parts][Hq][Lq][D] fp32 when parts > 1
  float* ws_lse;            // [parts][Hq][Lq] (log2 units)
  int Lq, T, S, cap, n_segs;
  int Hq, Hkv, D;
  int parts, n_rt;          // key-range parts, 256-row tiles of packed (token, head) rows
  int out_f32;
  float scale_log2;
};

struct AppendArgs {
  const uint16_t* kc;
  const uint16_t* vc;
  uint16_t* rk;
  uint16_t* rv;
  int C, R, p0;        // p0 = hist_len mod R
  int row_elems;       // Hkv * D
};

// The append of a chunk, ring[(p0 + j) mod R] <- chunk[j] for K and V, as
// 16-byte units: unit u in [0, 2*C*row_elems/8) (K units first, then V);
// threads take units first, first + stride, ...  Consecutive threads move
// consecutive units, so loads and stores are coalesced.
__device__ __forceinline__ void append_units(const AppendArgs& a, int64_t first, int64_t stride) {
  typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
  const int upt = a.row_elems >> 3;                  // 16-byte units per token row
  const int64_t per = (int64_t)a.C * upt;
  for (int64_t u = first; u < 2 * per; u += stride) {
    const bool v = u >= per;
    const int64_t w = v ? u - per : u;
    const int j = (int)(w / upt);
    const int c = (int)(w - (int64_t)j * upt);
    int slot = a.p0 + j;
    if (slot >= a.R) slot -= a.R;
    const uint16_t* src = v ? a.vc : a.kc;
    uint16_t* dst = v ? a.rv : a.rk;
    *(u32x4_t*)(dst + (int64_t)slot * a.row_elems + c * 8) = *(const u32x4_t*)(src + (int64_t)j * a.row_elems + c * 8);
  }
}

hipError_t launch_attention(const AttnArgs& a, int grid, hipStream_t stream);
// Merge of split key ranges (reads ws_o / ws_lse of `splits` parts, C rows per head).
hipError_t launch_merge(const AttnArgs& a, hipStream_t stream);
hipError_t launch_append(const AppendArgs& a, hipStream_t stream);
hipError_t launch_gather(const GatherArgs& a, hipStream_t stream);
// Records e as the calling thread's last HIP error; returns VICO_ERR_HIP.
int record_hip_failure(hipError_t e);

// Supplies a workspace of at least `need` bytes (address and size), or
// returns a negative vico_status.
using WorkspaceSource = int (*)(int64_t need, void** workspace, int64_t* workspace_bytes);

// Body of vico_gather_attn.  With `source` set, the workspace arguments are
// ignored when a workspace is needed: source() supplies it, and is called
// only after every other argument has been checked.
int gather_attn_entry(const void* q, int32_t q_len, const void* tail_k, const void* tail_v, int32_t tail_len,
                      const void* sink_k, const void* sink_v, int32_t sink_len, const void* store_k,
                      const void* store_v, int32_t store_slots, const int64_t* seg_start, const int32_t* seg_len,
                      int32_t num_segments, int64_t keys_hint, int32_t num_q_heads, int32_t num_kv_heads,
                      int32_t head_dim, float softmax_scale, void* out, int32_t out_dtype, float* lse_out,
                      int32_t num_splits, void* workspace, int64_t workspace_bytes, void* stream,
                      WorkspaceSource source);
hipError_t launch_token_mean(const uint16_t* x, int L, int dm, float* out, hipStream_t stream);
hipError_t launch_chunk_scores(const float* qf, const float* cf, int N, int dm, float* scores, hipStream_t stream);
hipError_t launch_topk(const float* scores, int N, int k, float min_score, const int64_t* chunk_start,
                       const int32_t* chunk_len, int32_t* out_chunks, float* out_scores, int64_t* seg_start,
                       int32_t* seg_len, int32_t* out_count, hipStream_t stream);

}  // namespace vico
