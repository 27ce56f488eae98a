// Chunk-level temporal token dropping for gfx950 (ViCoStream, Sec. 3,
// "Token Dropping").
//
// For every spatial position p of a chunk of C frames, the cosine of the
// projected tokens of every frame pair i < j is taken; the position is
// dropped when all of them exceed tau, and the first frame is kept as an
// anchor (frames 2..C lose their token at p).  With C = 1 each frame is
// compared with the frame before it (the previous chunk, or the caller's
// `prev` frame for the first one) and there is no anchor.
//
//   drop_sim_kernel<C>   one wave per (chunk, position): streams the C rows
//                        of dm bf16 once (16 bytes per lane per row per step),
//                        sums the C squared norms and C(C-1)/2 dot products
//                        in fp32, reduces them across the wave, and takes the
//                        decision in fp32 (the similarity it reports is the one
//                        the decision used).  HBM bound: reads the frames once.
//   drop_compact_kernel  one work-group per (chunk, 4-position tile): ranks
//                        its kept positions (counts of earlier chunks and
//                        positions, then a scan of the tile) and copies the
//                        retained token rows to their place in stream order.
//                        Reads the retained rows a second time and writes them
//                        once.
//   drop_fused_kernel    the single pass, taken when the caller supplies a
//                        workspace: the two steps above in one kernel, with
//                        every row read once (described further down).

#include "attn_common.h"
#include "token_drop.h"

#include <stdlib.h>

#include <algorithm>
#include <atomic>

namespace vico {
namespace {

constexpr int kDropThreads = 256;
constexpr int kCompactTile = 4;       // positions per compaction work-group (up to 32 rows to copy)
constexpr int kFusedMaxUnits = 8;     // single pass: rows of up to 8 * 64 * 8 = 4096 features
constexpr int kFusedMaxRegs = 128;    // single pass: row registers per lane, NV rows * units * 4
constexpr int kFusedMaxPositions = 1024;   // single pass: positions per frame (tiles per chunk <= 256)

__device__ __forceinline__ float wave_sum64(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Adds the products of one 16-byte unit (8 bf16 features) of NV vectors to
// the running fp32 norms and pair dots, in a fixed order; both schedules run
// this code, so their similarities are the same bits.
template <int NV, int NP>
__device__ __forceinline__ void sim_accumulate(const u32x4 (&v)[NV], float (&nrm)[NV], float (&dot)[NP]) {
  float x[NV][8];
#pragma unroll
  for (int f = 0; f < NV; ++f)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[f][2 * e] = __uint_as_float(v[f][e] << 16);
      x[f][2 * e + 1] = __uint_as_float(v[f][e] & 0xFFFF0000u);
    }
#pragma unroll
  for (int f = 0; f < NV; ++f)
#pragma unroll
    for (int e = 0; e < 8; ++e) nrm[f] += x[f][e] * x[f][e];
  int k = 0;
#pragma unroll
  for (int i = 0; i < NV; ++i)
#pragma unroll
    for (int j = i + 1; j < NV; ++j, ++k)
#pragma unroll
      for (int e = 0; e < 8; ++e) dot[k] += x[i][e] * x[j][e];
}

// Wave-wide sums of the partial norms and dots, every pair's cosine, and the
// decision: dropped when all of them exceed tau.  *smin receives the
// smallest cosine (the value the decision used).
template <int NV, int NP>
__device__ __forceinline__ bool sim_decide(float (&nrm)[NV], float (&dot)[NP], float tau, float* smin_out) {
#pragma unroll
  for (int f = 0; f < NV; ++f) nrm[f] = sqrtf(wave_sum64(nrm[f]));
#pragma unroll
  for (int k = 0; k < NP; ++k) dot[k] = wave_sum64(dot[k]);
  bool drop = true;
  float smin = INFINITY;
  int k = 0;
#pragma unroll
  for (int i = 0; i < NV; ++i)
#pragma unroll
    for (int j = i + 1; j < NV; ++j, ++k) {
      const float den = nrm[i] * nrm[j];
      const float s = den > 0.f ? dot[k] / den + 0.0f : 0.0f;   // + 0 turns -0 into +0
      drop = drop && (s > tau);
      smin = fminf(smin, s);
    }
  *smin_out = smin;
  return drop;
}

// The NV rows compared at position p of chunk b; vec[1] is null for the first
// frame of a C == 1 stream with no previous frame.
template <int C, int NV>
__device__ __forceinline__ void position_rows(const DropArgs& a, int b, int p, const uint16_t* (&vec)[NV]) {
  const int64_t dm = a.dm;
  if constexpr (C == 1) {
    vec[0] = a.frames + ((int64_t)b * a.n_f + p) * dm;
    vec[1] = b > 0 ? a.frames + ((int64_t)(b - 1) * a.n_f + p) * dm : (a.prev ? a.prev + (int64_t)p * dm : nullptr);
  } else {
#pragma unroll
    for (int f = 0; f < C; ++f) vec[f] = a.frames + (((int64_t)b * C + f) * a.n_f + p) * dm;
  }
}

template <int C>
__global__ __launch_bounds__(kDropThreads) void drop_sim_kernel(DropArgs a) {
  constexpr int NV = C == 1 ? 2 : C;            // vectors compared at one position
  constexpr int NP = NV * (NV - 1) / 2;         // pairs
  const int lane = threadIdx.x & 63;
  const int64_t item = ((int64_t)blockIdx.x * kDropThreads + threadIdx.x) >> 6;   // (chunk, position)
  if (item >= (int64_t)a.B * a.n_f) return;     // whole waves leave together
  const int b = (int)(item / a.n_f), p = (int)(item % a.n_f);
  const uint16_t* vec[NV];
  position_rows<C, NV>(a, b, p, vec);
  if (C == 1 && vec[1] == nullptr) {            // nothing before the first frame: kept
    if (lane == 0) {
      a.keep[item] = 1;
      if (a.sim) a.sim[item] = -2.0f;
    }
    return;
  }
  float nrm[NV], dot[NP];
#pragma unroll
  for (int f = 0; f < NV; ++f) nrm[f] = 0.f;
#pragma unroll
  for (int k = 0; k < NP; ++k) dot[k] = 0.f;
  for (int c8 = lane; c8 < a.dm / 8; c8 += 64) {
    u32x4 v[NV];
#pragma unroll
    for (int f = 0; f < NV; ++f) v[f] = *(const u32x4*)(vec[f] + c8 * 8);
    sim_accumulate<NV, NP>(v, nrm, dot);
  }
  float smin;
  const bool drop = sim_decide<NV, NP>(nrm, dot, a.tau, &smin);
  if (lane == 0) {
    a.keep[item] = drop ? 0 : 1;
    if (a.sim) a.sim[item] = smin;
  }
}

// Exclusive block-wide prefix sum over 256 threads; *total receives the sum.
__device__ __forceinline__ int scan256(int v, int* buf, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  if (lane == 63) buf[wave] = incl;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kDropThreads / 64; ++w) {
    base += w < wave ? buf[w] : 0;
    tot += buf[w];
  }
  __syncthreads();
  *total = tot;
  return base + incl - v;
}

// Kept flags in [lo, hi), summed over the work-group.
__device__ __forceinline__ int count_kept(const uint8_t* keep, int64_t lo, int64_t hi, int* buf) {
  int c = 0;
  for (int64_t i = lo + threadIdx.x; i < hi; i += kDropThreads) c += keep[i];
  int tot;
  scan256(c, buf, &tot);
  return tot;
}

__global__ __launch_bounds__(kDropThreads) void drop_compact_kernel(DropArgs a) {
  __shared__ int buf[kDropThreads / 64];
  __shared__ int row_src[8 * kCompactTile];     // flat source row of each retained token of the tile
  __shared__ int row_dst[8 * kCompactTile];
  static_assert(kCompactTile <= kDropThreads, "one thread per tile position");
  const int tid = threadIdx.x;
  const int tiles = (a.n_f + kCompactTile - 1) / kCompactTile;
  const int b = blockIdx.x / tiles;
  const int p0 = (blockIdx.x % tiles) * kCompactTile;
  const int np = min(kCompactTile, a.n_f - p0);
  const int C = a.C;
  const int anchor = C > 1 ? 1 : 0;              // frame 1 of every chunk is always kept
  const int m = C > 1 ? C - 1 : 1;               // frames that follow a position's flag
  const int64_t chunk0 = (int64_t)b * a.n_f;
  const int before = count_kept(a.keep, 0, chunk0, buf);               // kept positions of earlier chunks
  const int cnt_b = count_kept(a.keep, chunk0, chunk0 + a.n_f, buf);   // of this chunk
  const int pre = count_kept(a.keep, chunk0, chunk0 + p0, buf);        // of this chunk before the tile
  const int64_t base_b = (int64_t)b * anchor * a.n_f + (int64_t)m * before;   // first output row of chunk b
  const int flag = tid < np ? a.keep[chunk0 + p0 + tid] : 0;
  int tile_cnt;
  const int r = scan256(flag, buf, &tile_cnt);
  // list the tile's retained rows: frame f, position p0 + t
  if (tid < np) {
    const int p = p0 + tid;
    for (int f = 0; f < C; ++f) {
      const bool kept = (anchor && f == 0) || flag;
      if (!kept) continue;
      int64_t dst;
      int slot;
      if (anchor && f == 0) {
        dst = base_b + p;
        slot = tid;
      } else {
        dst = base_b + (int64_t)anchor * a.n_f + (int64_t)(f - anchor) * cnt_b + pre + r;
        slot = anchor * np + (f - anchor) * tile_cnt + r;
      }
      row_src[slot] = (int)(((int64_t)b * C + f) * a.n_f + p);
      row_dst[slot] = (int)dst;
    }
  }
  __syncthreads();
  const int n_rows = anchor * np + m * tile_cnt;
  for (int i = tid; i < n_rows; i += kDropThreads) a.out_index[row_dst[i]] = row_src[i];
  if (a.out) {
    // one wave per row; each lane loads all its 16-byte pieces of the row
    // (up to 8) before storing any, so a row's loads are in flight together
    const int ch = a.dm / 8;
    const int lane = tid & 63, wave = tid >> 6;
    for (int row = wave; row < n_rows; row += kDropThreads / 64) {
      const u32x4* __restrict__ src = (const u32x4*)(a.frames + (int64_t)row_src[row] * a.dm);
      u32x4* __restrict__ dst = (u32x4*)(a.out + (int64_t)row_dst[row] * a.dm);
      for (int c0 = 0; c0 < ch; c0 += 8 * 64) {
        u32x4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int c = c0 + k * 64 + lane;
          if (c < ch) v[k] = src[c];
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int c = c0 + k * 64 + lane;
          if (c < ch) dst[c] = v[k];
        }
      }
    }
  }
  if (b == a.B - 1 && p0 + np == a.n_f && tid == 0)
    a.out_count[0] = (int)(base_b + (int64_t)anchor * a.n_f + (int64_t)m * cnt_b);
}

// ---- single pass ---------------------------------------------------------
//
// One work-group per tile of kFusedWaves positions of one chunk (tile k =
// blockIdx.x is tile k % T of chunk k / T, T tiles per chunk), one wave per
// position.  The wave loads the NV rows of its position once, into registers,
// takes the decision with the arithmetic above, and later stores the retained
// rows straight to their place in stream order.  That place needs three
// counts of kept positions: of the chunk's tiles before this one (pre), of the
// whole chunk (cnt_b) and of all earlier chunks (before_b).  The groups share
// them through words in the workspace tagged with the call's epoch (a value
// the host never repeats), so nothing is zeroed between calls:
//   tile[k]   epoch << 3 | kept count of tile k;
//   chunk[b]  epoch << 12 | kept count of chunk b.
// The group of a chunk's last tile (its leader) reads the chunk's T tile
// words (up to 4 per lane) until all carry the epoch and publishes the chunk
// word; the other groups of the chunk wait for that one word, then read the
// words of the tiles before theirs.  Every group sums the chunk words before
// its chunk, 64 per read (one per lane).  A value read from another group sits
// inside one word, so relaxed atomics suffice: no cache write-back or
// invalidation, and no counter that all groups update.
// Waits are bounded in time (wait_ticks of the 100 MHz real-time counter).  A
// group whose wait runs out does not depend on the others any more: it
// recomputes the missing counts from the frames with the same arithmetic
// (same decisions, bit for bit) and reads its retained rows again, on a path
// where the rows held in registers are dead, so that path's registers do not
// add to the common path's (167 at 4 frames x 3584 features: three waves per
// SIMD).  The result therefore never depends on the order in which the
// hardware starts the groups; only the time does.  The epochs make a stale
// word from an earlier call unreadable as this call's (2^-52 odds for memory
// that never held one), and every store is bounds-checked, so a misread word
// could not send a row out of range.

constexpr int kFusedWaves = kDropThreads / 64;            // positions per work-group
constexpr int kFusedTileWords = 4;                        // tile words per lane: up to 256 tiles per chunk
constexpr int kFusedMaxChunks = 256;                      // chunks per call (a group reads all earlier chunk words)
static_assert(kFusedMaxPositions <= kFusedWaves * 64 * kFusedTileWords, "a wave reads all tile words of a chunk");

__host__ __device__ inline int drop_tiles_per_chunk(int n_f) { return (n_f + kFusedWaves - 1) / kFusedWaves; }

// Workspace layout: chunk[B] (one 128-byte line each: many groups read them),
// then tile[B * T], 8 bytes each.
__host__ __device__ inline int64_t drop_workspace_size(int B, int n_f) {
  return 128 * (int64_t)B + 8 * (int64_t)B * drop_tiles_per_chunk(n_f);
}

__device__ __forceinline__ unsigned long long load_word(const unsigned long long* w) {
  return __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_word(unsigned long long* w, unsigned long long v) {
  __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int wave_sum64_i32(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

struct Waiter {                       // a bounded wait: polls until the deadline passes
  uint64_t start, ticks;
  __device__ bool expired() const { return __builtin_amdgcn_s_memrealtime() - start > ticks; }
};

// The decision at position p of chunk b (1 = kept), taken by a whole wave
// from the frames.  Each accumulator receives the same products in the same
// order as in sim_accumulate (a lane's 16-byte units in turn, the 8 features
// of a unit in turn), so the decision is the same bit for bit; it reads two
// features of each row at a time to keep its registers few, since the rows of
// the group's own position stay live around it.
template <int C>
__device__ int decide_direct(const DropArgs& a, int b, int p) {
  constexpr int NV = C == 1 ? 2 : C;
  constexpr int NP = NV * (NV - 1) / 2;
  const int lane = threadIdx.x & 63;
  const uint16_t* vec[NV];
  position_rows<C, NV>(a, b, p, vec);
  if (C == 1 && vec[1] == nullptr) return 1;
  float nrm[NV], dot[NP];
#pragma unroll
  for (int f = 0; f < NV; ++f) nrm[f] = 0.f;
#pragma unroll
  for (int k = 0; k < NP; ++k) dot[k] = 0.f;
  for (int c8 = lane; c8 < a.dm / 8; c8 += 64) {
#pragma unroll 1
    for (int w = 0; w < 4; ++w) {
      float x[NV][2];
#pragma unroll
      for (int f = 0; f < NV; ++f) {
        const uint32_t v = *(const uint32_t*)(vec[f] + c8 * 8 + 2 * w);
        x[f][0] = __uint_as_float(v << 16);
        x[f][1] = __uint_as_float(v & 0xFFFF0000u);
      }
#pragma unroll
      for (int f = 0; f < NV; ++f)
#pragma unroll
        for (int e = 0; e < 2; ++e) nrm[f] += x[f][e] * x[f][e];
      int k = 0;
#pragma unroll
      for (int i = 0; i < NV; ++i)
#pragma unroll
        for (int j = i + 1; j < NV; ++j, ++k)
#pragma unroll
          for (int e = 0; e < 2; ++e) dot[k] += x[i][e] * x[j][e];
    }
  }
  float smin;
  return sim_decide<NV, NP>(nrm, dot, a.tau, &smin) ? 0 : 1;
}

// Kept positions of tiles [t_lo, t_hi) of chunk b from their words, waiting
// for them until the deadline.  Tiles still missing then are counted from the
// frames (RECOUNT), or the result is -1.  Run by a whole wave; the result is
// the same on every lane.
template <int C, bool RECOUNT>
__device__ int count_tiles(const DropArgs& a, const unsigned long long* tile, int b, int t_lo, int t_hi,
                           const Waiter& wt) {
  const int lane = threadIdx.x & 63;
  const int T = drop_tiles_per_chunk(a.n_f);
  const unsigned long long e = a.epoch;
  const unsigned long long* w = tile + (int64_t)b * T;
  unsigned missing;
  int sum;
  while (true) {
    missing = 0;
    sum = 0;
#pragma unroll
    for (int i = 0; i < kFusedTileWords; ++i) {
      const int k = t_lo + lane + 64 * i;
      if (k < t_hi) {
        const unsigned long long x = load_word(w + k);
        if ((x >> 3) == e) sum += min((int)(x & 7), kFusedWaves);
        else missing |= 1u << i;
      }
    }
    if (!__ballot(missing != 0)) return wave_sum64_i32(sum);
    if (wt.expired()) break;
    __builtin_amdgcn_s_sleep(2);
  }
  if constexpr (!RECOUNT) {
    return -1;
  } else {
    // recount the missing tiles, one position at a time across the wave
    for (int i = 0; i < kFusedTileWords; ++i) {
      unsigned long long todo = __ballot((missing >> i) & 1);
      while (todo) {
        const int l = __ffsll((long long)todo) - 1;
        todo &= todo - 1;
        const int k = t_lo + l + 64 * i;
        int c = 0;
        for (int q = k * kFusedWaves; q < min(a.n_f, (k + 1) * kFusedWaves); ++q) c += decide_direct<C>(a, b, q);
        if (lane == l) sum += c;
      }
    }
    return wave_sum64_i32(sum);
  }
}

// Kept positions of chunk b: its word, else (RECOUNT) its tiles, else -1.
template <int C, bool RECOUNT>
__device__ int count_chunk(const DropArgs& a, const unsigned long long* chunk, const unsigned long long* tile, int b,
                           const Waiter& wt) {
  const unsigned long long e = a.epoch;
  while (true) {
    const unsigned long long x = load_word(chunk + 16 * (int64_t)b);
    if ((x >> 12) == e) return min((int)(x & 0xFFF), a.n_f);
    if (wt.expired()) break;
    __builtin_amdgcn_s_sleep(2);
  }
  if constexpr (!RECOUNT) return -1;
  else return count_tiles<C, true>(a, tile, b, 0, drop_tiles_per_chunk(a.n_f), wt);
}

// Kept positions of chunks 0 .. b-1 (-1 as above); run by a whole wave.
template <int C, bool RECOUNT>
__device__ long long count_chunks_before(const DropArgs& a, const unsigned long long* chunk,
                                         const unsigned long long* tile, int b, const Waiter& wt) {
  const int lane = threadIdx.x & 63;
  const unsigned long long e = a.epoch;
  long long before = 0;
  for (int j0 = 0; j0 < b; j0 += 64) {
    const int j = j0 + lane;
    bool have = j >= b;
    int c = 0;
    while (true) {
      if (!have) {
        const unsigned long long x = load_word(chunk + 16 * (int64_t)j);
        if ((x >> 12) == e) {
          have = true;
          c = min((int)(x & 0xFFF), a.n_f);
        }
      }
      if (__ballot(!have) == 0 || wt.expired()) break;
      __builtin_amdgcn_s_sleep(2);
    }
    unsigned long long todo = __ballot(!have);
    if constexpr (!RECOUNT) {
      if (todo) return -1;
    } else {
      while (todo) {
        const int l = __ffsll((long long)todo) - 1;
        todo &= todo - 1;
        const int cc = count_tiles<C, true>(a, tile, j0 + l, 0, drop_tiles_per_chunk(a.n_f), wt);
        if (lane == l) c = cc;
      }
    }
    before += wave_sum64_i32(c);
  }
  return before;
}

// The three counts of tile (b, t) whose own count is tile_cnt; the chunk's
// leader (its last tile) publishes the chunk word.  Run by a whole wave.
// Without RECOUNT, false if a wait ran out.
template <int C, bool RECOUNT>
__device__ bool tile_counts(const DropArgs& a, unsigned long long* chunk, const unsigned long long* tile, int b, int t,
                            int tile_cnt, const Waiter& wt, int* pre_out, int* cnt_out, long long* before_out) {
  const int lane = threadIdx.x & 63;
  const int T = drop_tiles_per_chunk(a.n_f);
  int pre, cnt;
  if (t == T - 1) {
    pre = count_tiles<C, RECOUNT>(a, tile, b, 0, t, wt);
    if (pre < 0) return false;
    cnt = pre + tile_cnt;
    if (lane == 0) store_word(chunk + 16 * (int64_t)b, (a.epoch << 12) | (unsigned long long)cnt);
  } else {
    cnt = count_chunk<C, RECOUNT>(a, chunk, tile, b, wt);
    if (cnt < 0) return false;
    pre = count_tiles<C, RECOUNT>(a, tile, b, 0, t, wt);
    if (pre < 0) return false;
  }
  const long long before = count_chunks_before<C, RECOUNT>(a, chunk, tile, b, wt);
  if (before < 0) return false;
  *pre_out = pre;
  *cnt_out = cnt;
  *before_out = before;
  return true;
}

// Frames of a chunk kept whole (the anchor) and frames that follow a
// position's flag.
template <int C>
__device__ __forceinline__ int anchor_of() { return C > 1 ? 1 : 0; }
template <int C>
__device__ __forceinline__ int follow_of() { return C > 1 ? C - 1 : 1; }

// Output row of frame f at position p of a chunk whose first output row is
// base_b (cnt_b kept positions, rank kept positions of the chunk before p),
// or -1 where that token is dropped.
template <int C>
__device__ __forceinline__ int64_t retained_row(const DropArgs& a, int64_t base_b, int f, int p, int kept, int cnt_b,
                                                int rank) {
  const int anchor = anchor_of<C>();
  if (anchor && f == 0) return base_b + p;
  if (!kept) return -1;
  return base_b + (int64_t)anchor * a.n_f + (int64_t)(f - anchor) * cnt_b + rank;
}

// out_count, from the last chunk's counts.
template <int C>
__device__ __forceinline__ void drop_write_count(const DropArgs& a, long long before, int cnt) {
  __hip_atomic_store(a.out_count, (int)((int64_t)a.B * anchor_of<C>() * a.n_f + (int64_t)follow_of<C>() * (before + cnt)),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int C, int U>
__global__ __launch_bounds__(kDropThreads) void drop_fused_kernel(DropArgs a) {
  constexpr int NV = C == 1 ? 2 : C;
  constexpr int NP = NV * (NV - 1) / 2;
  __shared__ int s_ok, s_cnt, s_pre;
  __shared__ long long s_before;
  __shared__ int s_flag[kFusedWaves];
  const int T = drop_tiles_per_chunk(a.n_f);
  unsigned long long* chunk = (unsigned long long*)a.ws;  // one word per 128 bytes
  unsigned long long* tile = chunk + 16 * (int64_t)a.B;
  const unsigned long long e = a.epoch;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t tk = blockIdx.x;
  const int b = (int)(tk / T), t = (int)(tk - (int64_t)b * T);
  const int p0 = t * kFusedWaves;
  const int np = min(kFusedWaves, a.n_f - p0);
  const bool live = wave < np;
  const int p = live ? p0 + wave : p0;
  const int64_t chunk0 = (int64_t)b * a.n_f;
  const int dm8 = a.dm >> 3;

  // rows of the position, read once
  const uint16_t* vec[NV];
  position_rows<C, NV>(a, b, p, vec);
  const bool first = C == 1 && vec[1] == nullptr;         // no earlier frame: kept without comparison
  u32x4 x[NV][U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int c = u * 64 + lane;
#pragma unroll
    for (int f = 0; f < NV; ++f) {
      x[f][u] = u32x4{0u, 0u, 0u, 0u};
      if (live && c < dm8 && (f == 0 || !first)) x[f][u] = *(const u32x4*)(vec[f] + c * 8);
    }
  }

  int kept = 0;
  if (live) {
    if (first) {
      kept = 1;
      if (lane == 0 && a.sim) a.sim[chunk0 + p] = -2.0f;
    } else {
      float nrm[NV], dot[NP];
#pragma unroll
      for (int f = 0; f < NV; ++f) nrm[f] = 0.f;
#pragma unroll
      for (int k = 0; k < NP; ++k) dot[k] = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (u * 64 + lane < dm8) {
          u32x4 v[NV];
#pragma unroll
          for (int f = 0; f < NV; ++f) v[f] = x[f][u];
          sim_accumulate<NV, NP>(v, nrm, dot);
        }
      float smin;
      kept = sim_decide<NV, NP>(nrm, dot, a.tau, &smin) ? 0 : 1;
      if (lane == 0 && a.sim) a.sim[chunk0 + p] = smin;
    }
  }
  if (lane == 0) s_flag[wave] = kept;
  __syncthreads();

  // the three counts: shared by the other groups, or (slow path, below) recounted
  if (wave == 0) {
    int tile_cnt = 0;
    for (int i = 0; i < np; ++i) tile_cnt += s_flag[i];
    if (lane == 0) {
      for (int i = 0; i < np; ++i) a.keep[chunk0 + p0 + i] = (uint8_t)s_flag[i];
      store_word(tile + tk, (e << 3) | (unsigned long long)tile_cnt);
    }
    const Waiter wt{__builtin_amdgcn_s_memrealtime(), a.wait_ticks};
    int pre = 0, cnt = 0;
    long long before = 0;
    const bool ok = tile_counts<C, false>(a, chunk, tile, b, t, tile_cnt, wt, &pre, &cnt, &before);
    if (lane == 0) {
      s_ok = ok ? 1 : 0;
      s_before = before;
      s_pre = pre;
      s_cnt = cnt;
    }
  }
  __syncthreads();
  int r = 0;
  for (int i = 0; i < wave; ++i) r += s_flag[i];
  const int64_t rows = (int64_t)a.B * C * a.n_f;
  if (s_ok) {                                             // rows from registers
    if (tk == (int64_t)a.B * T - 1 && tid == 0) drop_write_count<C>(a, s_before, s_cnt);
    if (!live) return;
    const int64_t base_b = (int64_t)b * anchor_of<C>() * a.n_f + (int64_t)follow_of<C>() * s_before;
#pragma unroll
    for (int f = 0; f < C; ++f) {
      const int64_t dst = retained_row<C>(a, base_b, f, p, kept, s_cnt, s_pre + r);
      if (dst < 0 || dst >= rows) continue;               // dropped, or a misread word: never out of range
      if (lane == 0) a.out_index[dst] = (int)(((int64_t)b * C + f) * a.n_f + p);
      if (a.out) {
        u32x4* o = (u32x4*)(a.out + dst * a.dm);
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int c = u * 64 + lane;
          if (c < dm8) o[c] = x[f][u];
        }
      }
    }
    return;
  }
  // slow path: the rows in registers are dead here, which leaves the
  // registers to the recount; the retained rows are read again
  if (wave == 0) {
    const Waiter wt{0, 0};                                // already out of time
    int tile_cnt = 0;
    for (int i = 0; i < np; ++i) tile_cnt += s_flag[i];
    int pre = 0, cnt = 0;
    long long before = 0;
    tile_counts<C, true>(a, chunk, tile, b, t, tile_cnt, wt, &pre, &cnt, &before);
    if (lane == 0) {
      s_before = before;
      s_pre = pre;
      s_cnt = cnt;
    }
  }
  __syncthreads();
  if (tk == (int64_t)a.B * T - 1 && tid == 0) drop_write_count<C>(a, s_before, s_cnt);
  if (!live) return;
  const int64_t base_b = (int64_t)b * anchor_of<C>() * a.n_f + (int64_t)follow_of<C>() * s_before;
  for (int f = 0; f < C; ++f) {
    const int64_t dst = retained_row<C>(a, base_b, f, p, kept, s_cnt, s_pre + r);
    if (dst < 0 || dst >= rows) continue;
    const int64_t src = ((int64_t)b * C + f) * a.n_f + p;
    if (lane == 0) a.out_index[dst] = (int)src;
    if (a.out)
      for (int c = lane; c < dm8; c += 64) *(u32x4*)(a.out + dst * a.dm + c * 8) = *(const u32x4*)(a.frames + src * a.dm + c * 8);
  }
}

using FusedFn = void (*)(DropArgs);
template <int C, int U>
constexpr FusedFn fused_entry() {
  if constexpr ((C == 1 ? 2 : C) * U <= kFusedMaxRegs / 4) return drop_fused_kernel<C, U>;
  else return nullptr;
}
#define VICO_FUSED_ROW(C)                                                                                    \
  { fused_entry<C, 1>(), fused_entry<C, 2>(), fused_entry<C, 3>(), fused_entry<C, 4>(), fused_entry<C, 5>(), \
    fused_entry<C, 6>(), fused_entry<C, 7>(), fused_entry<C, 8>() }
const FusedFn kFused[8][kFusedMaxUnits] = {VICO_FUSED_ROW(1), VICO_FUSED_ROW(2), VICO_FUSED_ROW(3), VICO_FUSED_ROW(4),
                                           VICO_FUSED_ROW(5), VICO_FUSED_ROW(6), VICO_FUSED_ROW(7), VICO_FUSED_ROW(8)};
#undef VICO_FUSED_ROW

FusedFn fused_kernel_for(int B, int C, int n_f, int dm) {
  const int units = (dm / 8 + 63) / 64;                   // 16-byte pieces of a row per lane
  if (C < 1 || C > 8 || units > kFusedMaxUnits || n_f > kFusedMaxPositions || B > kFusedMaxChunks) return nullptr;
  return kFused[C - 1][units - 1];
}

// Per-call epochs: a bijection of a process-wide counter onto nonzero 52-bit
// values (odd multiplier and xor-shift modulo 2^52), so no two calls share one
// and they do not look like the small integers stale memory tends to hold.
uint64_t next_epoch() {
  static std::atomic<uint64_t> counter{0};
  constexpr uint64_t mask = (1ull << 52) - 1;
  uint64_t x = (counter.fetch_add(1, std::memory_order_relaxed) + 1) & mask;
  x = (x * 0x9E3779B97F4A7C15ull) & mask;
  x ^= x >> 26;
  x = (x * 0xBF58476D1CE4E5B9ull) & mask;
  x ^= x >> 23;
  return x;
}

// Longest wait for another group's count before recounting from the frames,
// in ticks of the 100 MHz real-time counter: 200 us, far above the wait of a
// whole call.  VICO_DROP_WAIT_US, read at every call, overrides it (tests set
// 0 to take the recounting path everywhere).
uint64_t wait_ticks() {
  const char* s = getenv("VICO_DROP_WAIT_US");
  const long us = s && *s ? strtol(s, nullptr, 10) : 200;
  return (uint64_t)(us < 0 ? 0 : us) * 100;
}

}  // namespace

int64_t temporal_drop_workspace_bytes(int B, int C, int n_f, int dm) {
  if (B < 1 || !fused_kernel_for(B, C, n_f, dm)) return 0;
  return drop_workspace_size(B, n_f);
}

hipError_t launch_temporal_drop(const DropArgs& a, hipStream_t stream) {
  const int64_t items = (int64_t)a.B * a.n_f;
  // single pass, except under graph capture: a replayed graph would repeat
  // the call's epoch and read the words of the previous replay as its own
  hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
  if (a.ws && hipStreamIsCapturing(stream, &capture) != hipSuccess) {
    (void)hipGetLastError();
    capture = hipStreamCaptureStatusActive;       // unknown: take the two passes
  }
  if (a.ws && capture == hipStreamCaptureStatusNone) {
    const FusedFn fn = fused_kernel_for(a.B, a.C, a.n_f, a.dm);
    if (!fn) return hipErrorInvalidValue;
    DropArgs args = a;
    args.epoch = next_epoch();
    args.wait_ticks = wait_ticks();
    void* kargs[] = {&args};
    return hipLaunchKernel((const void*)fn, dim3((unsigned)((int64_t)a.B * drop_tiles_per_chunk(a.n_f))),
                           dim3(kDropThreads), kargs, 0, stream);
  }
  const int blocks = (int)((items * 64 + kDropThreads - 1) / kDropThreads);
  switch (a.C) {
    case 1: hipLaunchKernelGGL(drop_sim_kernel<1>, dim3(blocks), dim3(kDropThreads), 0, stream, a); break;
    case 2: hipLaunchKernelGGL(drop_sim_kernel<2>, dim3(blocks), dim3(kDropThreads), 0, stream, a); break;
    case 3: hipLaunchKernelGGL(drop_sim_kernel<3>, dim3(blocks), dim3(kDropThreads), 0, stream, a); break;
    case 4: hipLaunchKernelGGL(drop_sim_kernel<4>, dim3(blocks), dim3(kDropThreads), 0, stream, a); break;
    case 5: hipLaunchKernelGGL(drop_sim_kernel<5>, dim3(blocks), dim3(kDropThreads), 0, stream, a); break;
    case 6: hipLaunchKernelGGL(drop_sim_kernel<6>, dim3(blocks), dim3(kDropThreads), 0, stream, a); break;
    case 7: hipLaunchKernelGGL(drop_sim_kernel<7>, dim3(blocks), dim3(kDropThreads), 0, stream, a); break;
    case 8: hipLaunchKernelGGL(drop_sim_kernel<8>, dim3(blocks), dim3(kDropThreads), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int tiles = (a.n_f + kCompactTile - 1) / kCompactTile;
  hipLaunchKernelGGL(drop_compact_kernel, dim3(a.B * tiles), dim3(kDropThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vico
