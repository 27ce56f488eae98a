// Host side of the C ABI declared in include/vico.h: argument validation,
// launch planning and error mapping.  Nothing here allocates device memory;
// every buffer, the workspace included, belongs to the caller.

#include <math.h>

#include <algorithm>
#include <stdint.h>

#include "vico.h"
#include "vico_internal.h"
#include "token_drop.h"

namespace {

thread_local int g_last_hip_error = 0;

constexpr int64_t kMaxChunk = int64_t(1) << 20;
constexpr int64_t kMaxKeys = int64_t(1) << 30;
constexpr int kMaxHeads = 1024;
constexpr int64_t kMaxTensorBytes = int64_t(1) << 31;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return na > 0 && nb > 0 && x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

struct Shape {
  int C, S, R, Wv, ws, Hq, Hkv, D, splits, balanced, grid, bidir, pack;
  int64_t total_tiles;
  int64_t ws_bytes;
};

int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// Row tiles of one head group: its C * pack packed rows ((token, query head)
// pairs, token-major) in blocks of kBlockM.
int64_t row_tiles(int C, int pack) { return (int64_t(C) * pack + vico::kBlockM - 1) / vico::kBlockM; }

// Key tiles of row tile rt: up to its last row's last visible key (the
// kernel's rule: the row's token position, or the chunk end when
// bidirectional).  The last row of row tile rt is token ((rt+1)*kBlockM-1)/pack.
int64_t tiles_of(int rt, int C, int SW, int bidir, int pack) {
  const int64_t last =
      bidir ? C : std::min<int64_t>((int64_t(rt + 1) * vico::kBlockM - 1) / pack + 1, C);
  return (SW + last + vico::kKeyTile - 1) / vico::kKeyTile;
}

// Splits of every row tile's key range: as many as keep the grid within one
// round of resident work-groups (so that, e.g., 48 row tiles take 5 splits
// and fill 240 of the 256 CUs), with at least kMinSplitTiles key tiles per
// split and at most kAutoSplits.
int plan_splits(int C, int S, int Wv, int Hq, int pack, int request) {
  const int64_t wgs = int64_t(Hq / pack) * row_tiles(C, pack);
  const int64_t tiles = (int64_t(S) + Wv + C + vico::kKeyTile - 1) / vico::kKeyTile;
  const int64_t cap = tiles < vico::kMaxSplits ? tiles : vico::kMaxSplits;
  if (request > 0) return (int)(request < cap ? request : cap);
  int64_t ns = int64_t(vico::kNumCUs) * vico::kWgPerCU / wgs;
  ns = std::min<int64_t>(std::min<int64_t>(ns, vico::kAutoSplits),
                         std::min<int64_t>(cap, tiles / vico::kMinSplitTiles));
  return (int)std::max<int64_t>(ns, 1);
}

// Balanced plan: gridDim.x equal shares of the (row tile, key tile) pairs.
// Returns the largest number of work-groups any row tile is spread over, or
// 0 when the balanced schedule does not apply.
int plan_balanced(int C, int SW, int Hq, int Hkv, int bidir, int pack, int64_t* total, int* grid) {
  const int n_rt = (int)row_tiles(C, pack);
  const int gq = Hq / Hkv / pack;
  int64_t T = 0;
  for (int rt = 0; rt < n_rt; ++rt) T += int64_t(Hq / pack) * tiles_of(rt, C, SW, bidir, pack);
  const int64_t G = int64_t(vico::kNumCUs) * vico::kWgPerCU;
  if (T < 4 * G) return 0;
  // walk the row tiles in kernel order: kv, row tile (longest first), head group
  int max_parts = 1;
  int64_t start = 0;
  for (int kv = 0; kv < Hkv; ++kv)
    for (int ri = 0; ri < n_rt; ++ri) {
      const int64_t n = tiles_of(n_rt - 1 - ri, C, SW, bidir, pack);
      for (int qh = 0; qh < gq; ++qh) {
        const int64_t w0 = ((start + 1) * G - 1) / T, w1 = ((start + n) * G - 1) / T;
        max_parts = (int)std::max<int64_t>(max_parts, w1 - w0 + 1);
        start += n;
      }
    }
  if (max_parts > vico::kMaxSplits) return 0;
  *total = T;
  *grid = (int)G;
  return max_parts;
}

// Validates everything the attention call and the planner share.
int check_attn_shape(int32_t C, int32_t S, int32_t R, int64_t H, int64_t W, int32_t Hq, int32_t Hkv,
                     int32_t D, int32_t splits, int32_t flags, Shape* sh) {
  if (C < 0 || S < 0 || R < 0 || H < 0 || W < -1 || splits < VICO_SPLIT_BALANCED) return VICO_ERR_INVALID_ARG;
  if (flags & ~(VICO_ATTN_BIDIRECTIONAL | VICO_ATTN_APPEND)) return VICO_ERR_INVALID_ARG;
  const int bidir = (flags & VICO_ATTN_BIDIRECTIONAL) ? 1 : 0;
  if (Hq < 1 || Hkv < 1 || Hq > kMaxHeads || Hq % Hkv != 0) return VICO_ERR_INVALID_ARG;
  if (D != 64 && D != 128) return VICO_ERR_UNSUPPORTED;
  if (C > kMaxChunk || S > kMaxChunk) return VICO_ERR_INVALID_ARG;
  const int64_t wv = (W < 0) ? H : (W < H ? W : H);
  if (wv > R) return VICO_ERR_CAPACITY;
  if (int64_t(S) + wv + C > kMaxKeys) return VICO_ERR_INVALID_ARG;
  // the kernels address every K/V tensor through 32-bit buffer offsets
  const int64_t row_bytes = int64_t(Hkv) * D * 2;
  if (row_bytes * C >= kMaxTensorBytes || row_bytes * S >= kMaxTensorBytes || row_bytes * R >= kMaxTensorBytes)
    return VICO_ERR_INVALID_ARG;
  sh->C = C; sh->S = S; sh->R = R; sh->Wv = (int)wv;
  sh->ws = R > 0 ? (int)((H - wv) % R) : 0;
  sh->Hq = Hq; sh->Hkv = Hkv; sh->D = D;
  sh->bidir = bidir;
  // Rows of a row tile: the tokens of one query head, or (token, query head)
  // pairs of all query heads of a KV head when that takes fewer row tiles --
  // a chunk of C tokens then leaves one part-filled row tile per KV head
  // instead of one per query head.
  sh->pack = row_tiles(C, Hq / Hkv) < int64_t(Hq / Hkv) * row_tiles(C, 1) ? Hq / Hkv : 1;
  sh->splits = 1;
  sh->balanced = 0;
  sh->total_tiles = 0;
  sh->grid = 0;
  if (C > 0) {
    const int64_t n_tiles_rows = int64_t(Hq / sh->pack) * row_tiles(C, sh->pack);   // row tiles, all heads
    const int ns = splits == VICO_SPLIT_BALANCED ? 1 : plan_splits(C, S, (int)wv, Hq, sh->pack, splits);
    int parts = 0;
    // balanced when asked for, or when the split grid would leave at least half
    // the CUs idle (measured: with most CUs busy the merge costs what the
    // balance gains -- the chip runs power-limited and idle CUs raise the clock)
    if (splits == VICO_SPLIT_BALANCED ||
        (splits == 0 && 2 * n_tiles_rows * ns <= int64_t(vico::kNumCUs) * vico::kWgPerCU))
      parts = plan_balanced(C, S + (int)wv, Hq, Hkv, bidir, sh->pack, &sh->total_tiles, &sh->grid);
    if (parts > 0) {
      sh->balanced = 1;
      sh->splits = parts;
    } else {
      sh->splits = ns;
      sh->grid = (int)(n_tiles_rows * ns);
    }
  }
  sh->ws_bytes = sh->splits > 1
                     ? align256(int64_t(4) * sh->splits * Hq * C * D) + int64_t(4) * sh->splits * Hq * C
                     : 0;
  return VICO_OK;
}

struct GatherShape {
  int Lq, T, S, cap, n_segs, Hq, Hkv, D, parts, n_rt;
  int64_t ws_bytes;
};

// Validates the shape arguments of the gathered attention and plans its
// key-range parts: enough work-groups to cover the CUs while every part keeps
// at least four key tiles of the expected key count.
int check_gather_shape(int32_t Lq, int32_t T, int32_t S, int32_t cap, int32_t n_segs, int64_t hint, int32_t Hq,
                       int32_t Hkv, int32_t D, int32_t splits, GatherShape* sh) {
  if (Lq < 0 || T < Lq || S < 0 || cap < 0 || n_segs < 0 || n_segs > vico::kMaxSegments || hint < 0 || splits < 0)
    return VICO_ERR_INVALID_ARG;
  if (Hq < 1 || Hkv < 1 || Hq > kMaxHeads || Hq % Hkv != 0) return VICO_ERR_INVALID_ARG;
  if (D != 64 && D != 128) return VICO_ERR_UNSUPPORTED;
  if (T > kMaxChunk || S > kMaxChunk) return VICO_ERR_INVALID_ARG;
  if (int64_t(n_segs) * cap + S + T > kMaxKeys) return VICO_ERR_INVALID_ARG;
  const int64_t row_bytes = int64_t(Hkv) * D * 2;
  if (row_bytes * T >= kMaxTensorBytes || row_bytes * S >= kMaxTensorBytes || row_bytes * cap >= kMaxTensorBytes ||
      int64_t(Lq) * Hq * D * 4 >= kMaxTensorBytes)
    return VICO_ERR_INVALID_ARG;
  const int g = Hq / Hkv;
  sh->Lq = Lq; sh->T = T; sh->S = S; sh->cap = cap; sh->n_segs = n_segs;
  sh->Hq = Hq; sh->Hkv = Hkv; sh->D = D;
  constexpr int kGatherRows = vico::kGatherThreads / 64 * 32;
  sh->n_rt = (int)((int64_t(g) * Lq + kGatherRows - 1) / kGatherRows);
  const int64_t tiles = (S + std::min<int64_t>(hint, kMaxKeys) + T + vico::kKeyTile - 1) / vico::kKeyTile;
  int parts = 1;
  if (splits > 0) {
    parts = std::min(splits, vico::kMaxGatherParts);
  } else {
    const int64_t base = int64_t(Hkv) * std::max(sh->n_rt, 1);
    while (parts * 2 <= vico::kMaxGatherParts && base * parts * 2 <= int64_t(vico::kNumCUs) * vico::kWgPerCU &&
           tiles >= 4 * int64_t(parts) * 2)
      parts *= 2;
  }
  sh->parts = parts;
  sh->ws_bytes = parts > 1 ? align256(int64_t(4) * parts * Hq * Lq * D) + int64_t(4) * parts * Hq * Lq : 0;
  return VICO_OK;
}

bool aligned_to(const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) & (n - 1)) == 0; }

int hip_fail(hipError_t e) {
  g_last_hip_error = (int)e;
  return VICO_ERR_HIP;
}

bool drop_shape_ok(int32_t num_chunks, int32_t frames_per_chunk, int32_t tokens_per_frame, int32_t feat_dim) {
  if (num_chunks < 0 || frames_per_chunk < 1 || frames_per_chunk > 8 || tokens_per_frame < 1 || feat_dim < 8 ||
      feat_dim % 8 != 0)
    return false;
  return int64_t(num_chunks) * frames_per_chunk * tokens_per_frame < (int64_t(1) << 31);
}

}  // namespace

int vico::record_hip_failure(hipError_t e) { return hip_fail(e); }

extern "C" {

const char* vico_status_str(int status) {
  switch (status) {
    case VICO_OK: return "ok";
    case VICO_ERR_INVALID_ARG: return "invalid argument";
    case VICO_ERR_UNSUPPORTED: return "unsupported head_dim or dtype";
    case VICO_ERR_CAPACITY: return "ring buffer too small for the window or the chunk";
    case VICO_ERR_MISALIGNED: return "pointer not 16-byte aligned";
    case VICO_ERR_WORKSPACE: return "workspace missing or too small";
    case VICO_ERR_HIP: return "HIP runtime error";
    case VICO_ERR_SCRATCH: return "call needs more than the library's fixed scratch array";
    default: return "unknown status";
  }
}

int vico_last_hip_error(void) { return g_last_hip_error; }

int vico_attn_plan(int32_t chunk_len, int32_t sink_len, int32_t ring_slots, int64_t hist_len, int64_t window,
                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, int32_t num_splits,
                   int32_t* num_splits_out, int64_t* workspace_bytes_out) {
  return vico_attn_plan_ex(chunk_len, sink_len, ring_slots, hist_len, window, num_q_heads, num_kv_heads, head_dim,
                           num_splits, 0, num_splits_out, workspace_bytes_out);
}

int vico_attn_plan_ex(int32_t chunk_len, int32_t sink_len, int32_t ring_slots, int64_t hist_len, int64_t window,
                      int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, int32_t num_splits, int32_t flags,
                      int32_t* num_splits_out, int64_t* workspace_bytes_out) {
  Shape sh;
  const int st = check_attn_shape(chunk_len, sink_len, ring_slots, hist_len, window, num_q_heads, num_kv_heads,
                                  head_dim, num_splits, flags, &sh);
  if (st != VICO_OK) return st;
  if (num_splits_out) *num_splits_out = sh.splits;
  if (workspace_bytes_out) *workspace_bytes_out = sh.ws_bytes;
  return VICO_OK;
}

int64_t vico_attn_workspace_bytes(int32_t chunk_len, int32_t sink_len, int32_t ring_slots, int64_t hist_len,
                                  int64_t window, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                  int32_t num_splits) {
  int64_t b = 0;
  const int st = vico_attn_plan(chunk_len, sink_len, ring_slots, hist_len, window, num_q_heads, num_kv_heads,
                                head_dim, num_splits, nullptr, &b);
  return st != VICO_OK ? int64_t(st) : b;
}

int vico_chunk_prefill_attn(const void* q, const void* k_chunk, const void* v_chunk, int32_t chunk_len,
                            const void* sink_k, const void* sink_v, int32_t sink_len, const void* ring_k,
                            const void* ring_v, int32_t ring_slots, int64_t hist_len, int64_t window,
                            int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float softmax_scale,
                            void* out, int32_t out_dtype, float* lse_out, int32_t num_splits, void* workspace,
                            int64_t workspace_bytes, void* stream) {
  return vico_chunk_prefill_attn_ex(q, k_chunk, v_chunk, chunk_len, sink_k, sink_v, sink_len, ring_k, ring_v,
                                    ring_slots, hist_len, window, num_q_heads, num_kv_heads, head_dim, softmax_scale,
                                    out, out_dtype, lse_out, num_splits, 0, workspace, workspace_bytes, stream);
}

int vico_chunk_prefill_attn_ex(const void* q, const void* k_chunk, const void* v_chunk, int32_t chunk_len,
                               const void* sink_k, const void* sink_v, int32_t sink_len, const void* ring_k,
                               const void* ring_v, int32_t ring_slots, int64_t hist_len, int64_t window,
                               int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float softmax_scale,
                               void* out, int32_t out_dtype, float* lse_out, int32_t num_splits, int32_t flags,
                               void* workspace, int64_t workspace_bytes, void* stream) {
  Shape sh;
  int st = check_attn_shape(chunk_len, sink_len, ring_slots, hist_len, window, num_q_heads, num_kv_heads, head_dim,
                            num_splits, flags, &sh);
  if (st != VICO_OK) return st;
  if (out_dtype != VICO_DTYPE_BF16 && out_dtype != VICO_DTYPE_F32) return VICO_ERR_UNSUPPORTED;
  if (isnan(softmax_scale) || isinf(softmax_scale)) return VICO_ERR_INVALID_ARG;
  if (workspace_bytes < 0) return VICO_ERR_INVALID_ARG;
  if (chunk_len == 0) return VICO_OK;
  if (!q || !k_chunk || !v_chunk || !out) return VICO_ERR_INVALID_ARG;
  if (sh.S > 0 && (!sink_k || !sink_v)) return VICO_ERR_INVALID_ARG;
  if (sh.Wv > 0 && (!ring_k || !ring_v)) return VICO_ERR_INVALID_ARG;
  const bool append = (flags & VICO_ATTN_APPEND) != 0;
  if (append && (!ring_k || !ring_v)) return VICO_ERR_INVALID_ARG;
  if (append && chunk_len > ring_slots) return VICO_ERR_CAPACITY;
  const void* ptrs[] = {q, k_chunk, v_chunk, sink_k, sink_v, ring_k, ring_v, out, workspace};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return VICO_ERR_MISALIGNED;
  if (lse_out && (reinterpret_cast<uintptr_t>(lse_out) & 3u)) return VICO_ERR_MISALIGNED;
  if (sh.ws_bytes > 0 && (!workspace || workspace_bytes < sh.ws_bytes)) return VICO_ERR_WORKSPACE;
  // The outputs must not alias any input.
  const int64_t ob = int64_t(chunk_len) * num_q_heads * head_dim * (out_dtype == VICO_DTYPE_F32 ? 4 : 2);
  const int64_t qb = int64_t(chunk_len) * num_q_heads * head_dim * 2;
  const int64_t cb = int64_t(chunk_len) * num_kv_heads * head_dim * 2;
  const int64_t sb = int64_t(sink_len) * num_kv_heads * head_dim * 2;
  const int64_t rb = int64_t(ring_slots) * num_kv_heads * head_dim * 2;
  const int64_t lb = lse_out ? int64_t(num_q_heads) * chunk_len * 4 : 0;
  const void* ins[] = {q, k_chunk, v_chunk, sink_k, sink_v, ring_k, ring_v};
  const int64_t inb[] = {qb, cb, cb, sb, sb, (sh.Wv || append) ? rb : 0, (sh.Wv || append) ? rb : 0};
  for (int i = 0; i < 7; ++i)
    if (ins[i] && (overlaps(out, ob, ins[i], inb[i]) || overlaps(lse_out, lb, ins[i], inb[i])))
      return VICO_ERR_INVALID_ARG;
  if (overlaps(out, ob, lse_out, lb)) return VICO_ERR_INVALID_ARG;
  // the append writes the ring: it must not alias the chunk, the other ring
  // tensor, or the workspace the merge reads in the same launch
  if (append) {
    const int64_t wsb = sh.splits > 1 ? sh.ws_bytes : 0;
    const void* other[] = {q, k_chunk, v_chunk, sink_k, sink_v, workspace};
    const int64_t otb[] = {qb, cb, cb, sb, sb, wsb};
    for (int i = 0; i < 6; ++i)
      if (other[i] && (overlaps(ring_k, rb, other[i], otb[i]) || overlaps(ring_v, rb, other[i], otb[i])))
        return VICO_ERR_INVALID_ARG;
    if (overlaps(ring_k, rb, ring_v, rb)) return VICO_ERR_INVALID_ARG;
  }

  vico::AttnArgs a{};
  a.q = (const uint16_t*)q;
  a.kc = (const uint16_t*)k_chunk;
  a.vc = (const uint16_t*)v_chunk;
  a.sink_k = (const uint16_t*)sink_k;
  a.sink_v = (const uint16_t*)sink_v;
  a.ring_k = (const uint16_t*)ring_k;
  a.ring_v = (const uint16_t*)ring_v;
  a.out = out;
  a.lse = lse_out;
  if (sh.splits > 1) {
    a.ws_o = (float*)workspace;
    a.ws_lse = (float*)((char*)workspace + align256(int64_t(4) * sh.splits * sh.Hq * sh.C * sh.D));
  }
  a.C = sh.C; a.S = sh.S; a.R = sh.R; a.Wv = sh.Wv; a.ws = sh.ws;
  a.Hq = sh.Hq; a.Hkv = sh.Hkv; a.D = sh.D;
  a.splits = sh.splits;
  a.balanced = sh.balanced;
  a.pack = sh.pack;
  a.total_tiles = sh.total_tiles;
  a.out_f32 = out_dtype == VICO_DTYPE_F32;
  a.bidir = sh.bidir;
  if (append) {
    a.app_rk = (uint16_t*)ring_k;
    a.app_rv = (uint16_t*)ring_v;
    a.app_p0 = (int)(hist_len % ring_slots);
  }
  const double scale = softmax_scale > 0.f ? double(softmax_scale) : 1.0 / sqrt(double(head_dim));
  a.scale_log2 = (float)(scale * 1.4426950408889634);
  const hipError_t e = vico::launch_attention(a, sh.grid, (hipStream_t)stream);
  return e == hipSuccess ? VICO_OK : hip_fail(e);
}

int64_t vico_acn_window(const int64_t* chunk_starts, int32_t num_chunks, int32_t t, int32_t acn) {
  if (!chunk_starts || num_chunks < 1 || t < 0 || t >= num_chunks) return VICO_ERR_INVALID_ARG;
  if (acn < 0) return chunk_starts[t];
  const int32_t first = t - acn > 0 ? t - acn : 0;
  const int64_t w = chunk_starts[t] - chunk_starts[first];
  return w < 0 ? int64_t(VICO_ERR_INVALID_ARG) : w;
}

int vico_kv_append(const void* k_chunk, const void* v_chunk, int32_t chunk_len, void* ring_k, void* ring_v,
                   int32_t ring_slots, int64_t hist_len, int32_t num_kv_heads, int32_t head_dim, void* stream) {
  if (chunk_len < 0 || ring_slots < 0 || hist_len < 0 || num_kv_heads < 1 || num_kv_heads > kMaxHeads)
    return VICO_ERR_INVALID_ARG;
  if (head_dim != 64 && head_dim != 128) return VICO_ERR_UNSUPPORTED;
  if (chunk_len > ring_slots) return VICO_ERR_CAPACITY;
  if (chunk_len == 0) return VICO_OK;
  if (!k_chunk || !v_chunk || !ring_k || !ring_v) return VICO_ERR_INVALID_ARG;
  const void* ptrs[] = {k_chunk, v_chunk, ring_k, ring_v};
  for (const void* p : ptrs)
    if (!aligned16(p)) return VICO_ERR_MISALIGNED;
  const int64_t row = int64_t(num_kv_heads) * head_dim * 2;
  const int64_t cb = row * chunk_len, rb = row * ring_slots;
  if (overlaps(ring_k, rb, ring_v, rb) || overlaps(ring_k, rb, k_chunk, cb) || overlaps(ring_k, rb, v_chunk, cb) ||
      overlaps(ring_v, rb, k_chunk, cb) || overlaps(ring_v, rb, v_chunk, cb))
    return VICO_ERR_INVALID_ARG;
  vico::AppendArgs a{};
  a.kc = (const uint16_t*)k_chunk;
  a.vc = (const uint16_t*)v_chunk;
  a.rk = (uint16_t*)ring_k;
  a.rv = (uint16_t*)ring_v;
  a.C = chunk_len;
  a.R = ring_slots;
  a.p0 = (int)(hist_len % ring_slots);
  a.row_elems = num_kv_heads * head_dim;
  const hipError_t e = vico::launch_append(a, (hipStream_t)stream);
  return e == hipSuccess ? VICO_OK : hip_fail(e);
}

int vico_token_mean(const void* x, int32_t num_tokens, int32_t feat_dim, float* out, void* stream) {
  if (num_tokens < 1 || feat_dim < 8 || feat_dim % 8 != 0) return VICO_ERR_INVALID_ARG;
  if (!x || !out) return VICO_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(out)) return VICO_ERR_MISALIGNED;
  if (overlaps(out, int64_t(feat_dim) * 4, x, int64_t(num_tokens) * feat_dim * 2)) return VICO_ERR_INVALID_ARG;
  const hipError_t e = vico::launch_token_mean((const uint16_t*)x, num_tokens, feat_dim, out, (hipStream_t)stream);
  return e == hipSuccess ? VICO_OK : hip_fail(e);
}

int vico_chunk_scores(const float* query_feat, const float* chunk_feat, int32_t num_chunks, int32_t feat_dim,
                      float* scores, void* stream) {
  if (num_chunks < 0 || feat_dim < 8 || feat_dim % 8 != 0) return VICO_ERR_INVALID_ARG;
  if (num_chunks == 0) return VICO_OK;
  if (!query_feat || !chunk_feat || !scores) return VICO_ERR_INVALID_ARG;
  if (!aligned16(query_feat) || !aligned16(chunk_feat) || !aligned_to(scores, 4)) return VICO_ERR_MISALIGNED;
  const int64_t fb = int64_t(num_chunks) * feat_dim * 4;
  if (overlaps(scores, int64_t(num_chunks) * 4, chunk_feat, fb) ||
      overlaps(scores, int64_t(num_chunks) * 4, query_feat, int64_t(feat_dim) * 4))
    return VICO_ERR_INVALID_ARG;
  const hipError_t e = vico::launch_chunk_scores(query_feat, chunk_feat, num_chunks, feat_dim, scores,
                                                 (hipStream_t)stream);
  return e == hipSuccess ? VICO_OK : hip_fail(e);
}

int vico_topk_chunks(const float* scores, int32_t num_chunks, int32_t top_k, float min_score,
                     const int64_t* chunk_start, const int32_t* chunk_len, int32_t* out_chunks,
                     float* out_scores, int64_t* seg_start, int32_t* seg_len, int32_t* out_count, void* stream) {
  if (num_chunks < 0 || top_k < 1 || top_k > vico::kMaxSegments || isnan(min_score)) return VICO_ERR_INVALID_ARG;
  if ((num_chunks > 0 && !scores) || !out_chunks || !out_scores || !out_count) return VICO_ERR_INVALID_ARG;
  const bool segs = chunk_start || chunk_len;
  if (segs && (!chunk_start || !chunk_len || !seg_start || !seg_len)) return VICO_ERR_INVALID_ARG;
  if (!aligned_to(scores, 4) || !aligned_to(out_chunks, 4) || !aligned_to(out_scores, 4) ||
      !aligned_to(out_count, 4) || !aligned_to(chunk_start, 8) || !aligned_to(chunk_len, 4) ||
      !aligned_to(seg_start, 8) || !aligned_to(seg_len, 4))
    return VICO_ERR_MISALIGNED;
  const int64_t kb4 = int64_t(top_k) * 4;
  const void* outs[] = {out_chunks, out_scores, out_count, segs ? (const void*)seg_start : nullptr,
                        segs ? (const void*)seg_len : nullptr};
  const int64_t outb[] = {kb4, kb4, 4, 2 * kb4, kb4};
  const void* ins[] = {scores, chunk_start, chunk_len};
  const int64_t inb[] = {int64_t(num_chunks) * 4, int64_t(num_chunks) * 8, int64_t(num_chunks) * 4};
  for (int i = 0; i < 5; ++i) {
    if (!outs[i]) continue;
    for (int j = 0; j < 3; ++j)
      if (ins[j] && overlaps(outs[i], outb[i], ins[j], inb[j])) return VICO_ERR_INVALID_ARG;
    for (int j = i + 1; j < 5; ++j)
      if (outs[j] && overlaps(outs[i], outb[i], outs[j], outb[j])) return VICO_ERR_INVALID_ARG;
  }
  const hipError_t e = vico::launch_topk(scores, num_chunks, top_k, min_score, segs ? chunk_start : nullptr,
                                         chunk_len, out_chunks, out_scores, segs ? seg_start : nullptr, seg_len,
                                         out_count, (hipStream_t)stream);
  return e == hipSuccess ? VICO_OK : hip_fail(e);
}

int vico_gather_plan(int32_t q_len, int32_t tail_len, int32_t sink_len, int32_t store_slots, int32_t num_segments,
                     int64_t keys_hint, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                     int32_t num_splits, int32_t* num_splits_out, int64_t* workspace_bytes_out) {
  GatherShape sh;
  const int st = check_gather_shape(q_len, tail_len, sink_len, store_slots, num_segments, keys_hint, num_q_heads,
                                    num_kv_heads, head_dim, num_splits, &sh);
  if (st != VICO_OK) return st;
  if (num_splits_out) *num_splits_out = sh.parts;
  if (workspace_bytes_out) *workspace_bytes_out = sh.ws_bytes;
  return VICO_OK;
}

int vico_gather_attn(const void* q, int32_t q_len, const void* tail_k, const void* tail_v, int32_t tail_len,
                     const void* sink_k, const void* sink_v, int32_t sink_len, const void* store_k,
                     const void* store_v, int32_t store_slots, const int64_t* seg_start, const int32_t* seg_len,
                     int32_t num_segments, int64_t keys_hint, int32_t num_q_heads, int32_t num_kv_heads,
                     int32_t head_dim, float softmax_scale, void* out, int32_t out_dtype, float* lse_out,
                     int32_t num_splits, void* workspace, int64_t workspace_bytes, void* stream) {
  return vico::gather_attn_entry(q, q_len, tail_k, tail_v, tail_len, sink_k, sink_v, sink_len, store_k, store_v,
                                 store_slots, seg_start, seg_len, num_segments, keys_hint, num_q_heads,
                                 num_kv_heads, head_dim, softmax_scale, out, out_dtype, lse_out, num_splits,
                                 workspace, workspace_bytes, stream, nullptr);
}

}  // extern "C"

int vico::gather_attn_entry(const void* q, int32_t q_len, const void* tail_k, const void* tail_v, int32_t tail_len,
                            const void* sink_k, const void* sink_v, int32_t sink_len, const void* store_k,
                            const void* store_v, int32_t store_slots, const int64_t* seg_start,
                            const int32_t* seg_len, int32_t num_segments, int64_t keys_hint, int32_t num_q_heads,
                            int32_t num_kv_heads, int32_t head_dim, float softmax_scale, void* out,
                            int32_t out_dtype, float* lse_out, int32_t num_splits, void* workspace,
                            int64_t workspace_bytes, void* stream, WorkspaceSource source) {
  GatherShape sh;
  int st = check_gather_shape(q_len, tail_len, sink_len, store_slots, num_segments, keys_hint, num_q_heads,
                              num_kv_heads, head_dim, num_splits, &sh);
  if (st != VICO_OK) return st;
  if (out_dtype != VICO_DTYPE_BF16 && out_dtype != VICO_DTYPE_F32) return VICO_ERR_UNSUPPORTED;
  if (isnan(softmax_scale) || isinf(softmax_scale)) return VICO_ERR_INVALID_ARG;
  if (workspace_bytes < 0) return VICO_ERR_INVALID_ARG;
  if (q_len == 0) return VICO_OK;
  if (!q || !tail_k || !tail_v || !out) return VICO_ERR_INVALID_ARG;
  if (sink_len > 0 && (!sink_k || !sink_v)) return VICO_ERR_INVALID_ARG;
  if (num_segments > 0 && (!seg_start || !seg_len)) return VICO_ERR_INVALID_ARG;
  if (num_segments > 0 && store_slots > 0 && (!store_k || !store_v)) return VICO_ERR_INVALID_ARG;
  const void* ptrs[] = {q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, out, workspace};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return VICO_ERR_MISALIGNED;
  if (!aligned_to(seg_start, 8) || !aligned_to(seg_len, 4) || !aligned_to(lse_out, 4)) return VICO_ERR_MISALIGNED;
  const int64_t ob = int64_t(q_len) * num_q_heads * head_dim * (out_dtype == VICO_DTYPE_F32 ? 4 : 2);
  const int64_t row = int64_t(num_kv_heads) * head_dim * 2;
  const int64_t lb = lse_out ? int64_t(num_q_heads) * q_len * 4 : 0;
  const void* ins[] = {q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len};
  const int64_t inb[] = {int64_t(q_len) * num_q_heads * head_dim * 2, row * tail_len, row * tail_len,
                         row * sink_len, row * sink_len, row * store_slots, row * store_slots,
                         int64_t(num_segments) * 8, int64_t(num_segments) * 4};
  for (int i = 0; i < 9; ++i)
    if (ins[i] && (overlaps(out, ob, ins[i], inb[i]) || overlaps(lse_out, lb, ins[i], inb[i])))
      return VICO_ERR_INVALID_ARG;
  if (overlaps(out, ob, lse_out, lb)) return VICO_ERR_INVALID_ARG;
  // the library's own workspace is looked up only for a call known to be valid
  if (source && sh.ws_bytes > 0) {
    st = source(sh.ws_bytes, &workspace, &workspace_bytes);
    if (st != VICO_OK) return st;
  }
  if (sh.ws_bytes > 0 && (!workspace || workspace_bytes < sh.ws_bytes)) return VICO_ERR_WORKSPACE;

  vico::GatherArgs a{};
  a.q = (const uint16_t*)q;
  a.tail_k = (const uint16_t*)tail_k;
  a.tail_v = (const uint16_t*)tail_v;
  a.sink_k = (const uint16_t*)sink_k;
  a.sink_v = (const uint16_t*)sink_v;
  a.store_k = (const uint16_t*)store_k;
  a.store_v = (const uint16_t*)store_v;
  a.seg_start = seg_start;
  a.seg_len = seg_len;
  a.out = out;
  a.lse = lse_out;
  if (sh.parts > 1) {
    a.ws_o = (float*)workspace;
    a.ws_lse = (float*)((char*)workspace + align256(int64_t(4) * sh.parts * sh.Hq * sh.Lq * sh.D));
  }
  a.Lq = sh.Lq; a.T = sh.T; a.S = sh.S;
  a.cap = (store_k && store_v) ? sh.cap : 0;
  a.n_segs = sh.n_segs;
  a.Hq = sh.Hq; a.Hkv = sh.Hkv; a.D = sh.D;
  a.parts = sh.parts;
  a.n_rt = sh.n_rt;
  a.out_f32 = out_dtype == VICO_DTYPE_F32;
  const double scale = softmax_scale > 0.f ? double(softmax_scale) : 1.0 / sqrt(double(head_dim));
  a.scale_log2 = (float)(scale * 1.4426950408889634);
  const hipError_t e = vico::launch_gather(a, (hipStream_t)stream);
  return e == hipSuccess ? VICO_OK : hip_fail(e);
}

extern "C" {

int64_t vico_temporal_drop_workspace_bytes(int32_t num_chunks, int32_t frames_per_chunk, int32_t tokens_per_frame,
                                           int32_t feat_dim) {
  if (!drop_shape_ok(num_chunks, frames_per_chunk, tokens_per_frame, feat_dim)) return VICO_ERR_INVALID_ARG;
  return vico::temporal_drop_workspace_bytes(num_chunks, frames_per_chunk, tokens_per_frame, feat_dim);
}

int vico_temporal_drop(const void* frames, int32_t num_chunks, int32_t frames_per_chunk, int32_t tokens_per_frame,
                       int32_t feat_dim, float tau, const void* prev_frame, uint8_t* keep, float* sim,
                       void* out_tokens, int32_t* out_index, int32_t* out_count, void* workspace,
                       int64_t workspace_bytes, void* stream) {
  if (!drop_shape_ok(num_chunks, frames_per_chunk, tokens_per_frame, feat_dim) || isnan(tau) || workspace_bytes < 0)
    return VICO_ERR_INVALID_ARG;
  const int64_t rows = int64_t(num_chunks) * frames_per_chunk * tokens_per_frame;
  if (num_chunks == 0) return VICO_OK;
  if (!frames || !keep || !out_index || !out_count) return VICO_ERR_INVALID_ARG;
  const int64_t need = workspace ? vico::temporal_drop_workspace_bytes(num_chunks, frames_per_chunk, tokens_per_frame,
                                                                       feat_dim) : 0;
  if (!aligned16(frames) || (prev_frame && !aligned16(prev_frame)) || (out_tokens && !aligned16(out_tokens)) ||
      !aligned_to(sim, 4) || !aligned_to(out_index, 4) || !aligned_to(out_count, 4) ||
      (need && !aligned_to(workspace, 8)))
    return VICO_ERR_MISALIGNED;
  const int64_t fb = rows * feat_dim * 2, pb = prev_frame ? int64_t(tokens_per_frame) * feat_dim * 2 : 0;
  const int64_t kb = int64_t(num_chunks) * tokens_per_frame;
  const void* outs[] = {keep, sim, out_tokens, out_index, out_count, need ? workspace : nullptr};
  const int64_t outb[] = {kb, sim ? kb * 4 : 0, out_tokens ? fb : 0, rows * 4, 4, need};
  for (int i = 0; i < 6; ++i) {
    if (!outs[i]) continue;
    if (overlaps(outs[i], outb[i], frames, fb) || overlaps(outs[i], outb[i], prev_frame, pb)) return VICO_ERR_INVALID_ARG;
    for (int j = i + 1; j < 6; ++j)
      if (outs[j] && overlaps(outs[i], outb[i], outs[j], outb[j])) return VICO_ERR_INVALID_ARG;
  }
  if (need && workspace_bytes < need) return VICO_ERR_WORKSPACE;
  vico::DropArgs a{};
  a.ws = need ? workspace : nullptr;
  a.frames = (const uint16_t*)frames;
  a.prev = frames_per_chunk == 1 ? (const uint16_t*)prev_frame : nullptr;
  a.keep = keep;
  a.sim = sim;
  a.out = (uint16_t*)out_tokens;
  a.out_index = out_index;
  a.out_count = out_count;
  a.B = num_chunks;
  a.C = frames_per_chunk;
  a.n_f = tokens_per_frame;
  a.dm = feat_dim;
  a.tau = tau;
  const hipError_t e = vico::launch_temporal_drop(a, (hipStream_t)stream);
  return e == hipSuccess ? VICO_OK : hip_fail(e);
}

}  // extern "C"
