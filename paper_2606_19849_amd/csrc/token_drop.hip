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
//                        Reads the retained rows a second time (mostly from L2)
//                        and writes them once.

#include "attn_common.h"

namespace vico {
namespace {

constexpr int kDropThreads = 256;
constexpr int kCompactTile = 4;       // positions per compaction work-group (up to 32 rows to copy)

__device__ __forceinline__ float wave_sum64(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <int C>
__global__ __launch_bounds__(kDropThreads) void drop_sim_kernel(DropArgs a) {
  constexpr int NV = C == 1 ? 2 : C;            // vectors compared at one position
  constexpr int NP = NV * (NV - 1) / 2;         // pairs
  const int lane = threadIdx.x & 63;
  const int64_t item = ((int64_t)blockIdx.x * kDropThreads + threadIdx.x) >> 6;   // (chunk, position)
  if (item >= (int64_t)a.B * a.n_f) return;     // whole waves leave together
  const int b = (int)(item / a.n_f), p = (int)(item % a.n_f);
  const int64_t dm = a.dm;
  const uint16_t* vec[NV];
  if constexpr (C == 1) {
    vec[0] = a.frames + ((int64_t)b * a.n_f + p) * dm;
    vec[1] = b > 0 ? a.frames + ((int64_t)(b - 1) * a.n_f + p) * dm : (a.prev ? a.prev + (int64_t)p * dm : nullptr);
    if (vec[1] == nullptr) {                    // nothing before the first frame: kept
      if (lane == 0) {
        a.keep[item] = 1;
        if (a.sim) a.sim[item] = -2.0f;
      }
      return;
    }
  } else {
#pragma unroll
    for (int f = 0; f < C; ++f) vec[f] = a.frames + (((int64_t)b * C + f) * a.n_f + p) * dm;
  }
  float nrm[NV], dot[NP];
#pragma unroll
  for (int f = 0; f < NV; ++f) nrm[f] = 0.f;
#pragma unroll
  for (int k = 0; k < NP; ++k) dot[k] = 0.f;
  for (int c8 = lane; c8 < a.dm / 8; c8 += 64) {
    float x[NV][8];
#pragma unroll
    for (int f = 0; f < NV; ++f) {
      const u32x4 v = *(const u32x4*)(vec[f] + c8 * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[f][2 * e] = __uint_as_float(v[e] << 16);
        x[f][2 * e + 1] = __uint_as_float(v[e] & 0xFFFF0000u);
      }
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
      drop = drop && (s > a.tau);
      smin = fminf(smin, s);
    }
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

}  // namespace

hipError_t launch_temporal_drop(const DropArgs& a, hipStream_t stream) {
  const int64_t items = (int64_t)a.B * a.n_f;
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
