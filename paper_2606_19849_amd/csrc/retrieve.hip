// Query-side chunk retrieval for gfx950: representative features, cosine
// scores and top-k selection (ViCoStream, Sec. 3, query-time decoding).
//
//   token_mean_kernel   mean over tokens of a [L][dm] bf16 embedding block,
//                       fp32 out (a chunk's feature at ingest, or the query's)
//   chunk_scores_kernel s_i = <q, c_i> / (|q| |c_i|) over the feature table
//   topk_kernel         the k best chunks with s >= tau_q (ties: smaller
//                       index), written in stream order together with their
//                       store segments, for the gathered attention
//
// All three are bound by HBM or by launch latency; none of them needs a
// workspace.  Every reduction runs in a fixed order, so results repeat
// bit for bit.

#include "attn_common.h"

namespace vico {
namespace {

constexpr int kMeanThreads = 1024;   // 16 waves split the tokens; 4 columns per lane
constexpr int kMeanCols = 256;       // columns per work-group
constexpr int kTopkThreads = 1024;
constexpr int kTopkRegKeys = 8;      // scores kept in registers per thread (N <= 8192 read once)

__global__ __launch_bounds__(kMeanThreads) void token_mean_kernel(const uint16_t* __restrict__ x, int L, int dm,
                                                                  float* __restrict__ out) {
  constexpr int NW = kMeanThreads / 64;
  __shared__ f32x4 part[NW][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.x * kMeanCols + lane * 4;
  f32x4 acc{0.f, 0.f, 0.f, 0.f};
  if (col < dm) {
    const uint16_t* p = x + col;
    for (int t = wave; t < L; t += NW) {
      const uint2 v = *(const uint2*)(p + (int64_t)t * dm);
      acc[0] += __uint_as_float(v.x << 16);
      acc[1] += __uint_as_float(v.x & 0xFFFF0000u);
      acc[2] += __uint_as_float(v.y << 16);
      acc[3] += __uint_as_float(v.y & 0xFFFF0000u);
    }
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && col < dm) {
    f32x4 s = part[0][lane];
    for (int w = 1; w < NW; ++w) s += part[w][lane];
    *(f32x4*)(out + col) = f32x4{s[0] / (float)L, s[1] / (float)L, s[2] / (float)L, s[3] / (float)L};
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// One wave per chunk (grid-stride over chunks).  |q|^2, <q, c_i> and |c_i|^2
// are summed in one walk over the features, kScoreBatch float4 of q and of
// the row per lane loaded before any is used, so a 3584-feature row costs two
// memory latencies.  Each lane adds its columns in increasing order and the
// wave reduction is fixed, so every wave gets the same |q|^2 bits.
constexpr int kScoreBatch = 8;
__global__ __launch_bounds__(256) void chunk_scores_kernel(const float* __restrict__ qf, const float* __restrict__ cf,
                                                           int N, int dm, float* __restrict__ scores) {
  const int lane = threadIdx.x & 63;
  const int gw = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int nw = (gridDim.x * blockDim.x) >> 6;
  const int n4 = dm / 4;
  for (int i = gw; i < N; i += nw) {
    const float* row = cf + (int64_t)i * dm;
    float dot = 0.f, cc = 0.f, qq = 0.f;
    for (int c0 = lane; c0 < n4; c0 += 64 * kScoreBatch) {
      f32x4 q[kScoreBatch], v[kScoreBatch];
#pragma unroll
      for (int u = 0; u < kScoreBatch; ++u) {
        const int c = min(c0 + 64 * u, n4 - 1);      // in range; the sums below skip c >= n4
        q[u] = *(const f32x4*)(qf + 4 * c);
        v[u] = *(const f32x4*)(row + 4 * c);
      }
#pragma unroll
      for (int u = 0; u < kScoreBatch; ++u)
        if (c0 + 64 * u < n4) {
          qq += q[u][0] * q[u][0] + q[u][1] * q[u][1] + q[u][2] * q[u][2] + q[u][3] * q[u][3];
          dot += q[u][0] * v[u][0] + q[u][1] * v[u][1] + q[u][2] * v[u][2] + q[u][3] * v[u][3];
          cc += v[u][0] * v[u][0] + v[u][1] * v[u][1] + v[u][2] * v[u][2] + v[u][3] * v[u][3];
        }
    }
    qq = wave_sum(qq);
    dot = wave_sum(dot);
    cc = wave_sum(cc);
    if (lane == 0) {
      const float den = sqrtf(cc) * sqrtf(qq);
      scores[i] = den > 0.f ? dot / den + 0.0f : 0.0f;   // + 0 turns -0 into +0
    }
  }
}

// Order-preserving map of a (non-NaN) float to an unsigned key.
__device__ __forceinline__ uint32_t order_key(float s) {
  const uint32_t u = __float_as_uint(s + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

struct TopkArgs {
  const float* scores;
  int N, k;
  float min_score;
  const int64_t* chunk_start;
  const int32_t* chunk_len;
  int32_t* out_chunks;
  float* out_scores;
  int64_t* seg_start;
  int32_t* seg_len;
  int32_t* out_count;
};

// Exclusive block-wide prefix sum of v (NT threads); *total gets the sum.
// `buf` holds one slot per wave; the caller separates successive calls with
// a barrier (done at the end here).
template <int NT>
__device__ __forceinline__ int block_scan(int v, int* buf, int* total) {
  constexpr int NW = NT / 64;
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
  for (int w = 0; w < NW; ++w) {
    const int t = buf[w];
    base += w < wave ? t : 0;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return base + incl - v;
}

// NT threads: 256 for up to 256 scores (fewer waves to synchronise at each
// of the select's barriers), else 1024.
template <int NT>
__global__ __launch_bounds__(NT) void topk_kernel(TopkArgs a) {
  static_assert(NT >= 256, "one thread per histogram bin");
  constexpr int NR = kTopkRegKeys;
  __shared__ int hist[256];
  __shared__ int scan_buf[NT / 64];
  __shared__ int sh_bin, sh_remaining;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // key of score i, 0 for "not a candidate" (0 is the key of a NaN pattern,
  // which is never a candidate)
  auto key_of = [&](int i) __attribute__((always_inline)) -> uint32_t {
    const float s = a.scores[i];
    return (!isnan(s) && s >= a.min_score) ? order_key(s) : 0u;
  };
  // the first NR * NT keys stay in registers; the rest are re-read
  uint32_t kr[NR];
#pragma unroll
  for (int j = 0; j < NR; ++j) {
    const int i = tid + j * NT;
    kr[j] = i < a.N ? key_of(i) : 0u;
  }
  auto for_each_key = [&](auto&& fn) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < NR; ++j) fn(kr[j]);
    for (int i = tid + NR * NT; i < a.N; i += NT) fn(key_of(i));
  };

  int cnt = 0;
  for_each_key([&](uint32_t k) __attribute__((always_inline)) { cnt += k != 0u; });
  int n_cand;
  block_scan<NT>(cnt, scan_buf, &n_cand);
  const bool take_all = n_cand <= a.k;

  // radix select of the k-th largest key, 8 bits at a time from the top
  uint32_t prefix = 0, mask = 0;
  int remaining = a.k;
  if (!take_all) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (tid < 256) hist[tid] = 0;
      __syncthreads();
      for_each_key([&](uint32_t k) __attribute__((always_inline)) {
        if (k != 0u && (k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1);
      });
      __syncthreads();
      if (wave == 0) {
        // lane l holds bins 255-4l .. 252-4l; find the bin where the count of
        // keys from the top first reaches `remaining`
        int c[4], tot = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) { c[e] = hist[255 - 4 * lane - e]; tot += c[e]; }
        int incl = tot;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(incl, o, 64);
          if (lane >= o) incl += y;
        }
        int cum = incl - tot;
        if (cum < remaining && incl >= remaining) {
          int e_hit = 3, cum_hit = cum;
          bool found = false;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (!found && cum + c[e] >= remaining) { found = true; e_hit = e; cum_hit = cum; }
            cum += c[e];
          }
          sh_bin = 255 - 4 * lane - e_hit;
          sh_remaining = remaining - cum_hit;
        }
      }
      __syncthreads();
      prefix |= (uint32_t)sh_bin << shift;
      mask |= 255u << shift;
      remaining = sh_remaining;
    }
  }
  // prefix = key of the k-th best; keys above it are all taken, and
  // `remaining` of those equal to it, earliest first

  int taken = 0, eq_seen = 0;
  auto emit = [&](int i, uint32_t key) __attribute__((always_inline)) {
    const bool cand = key != 0u;
    const bool gt = cand && (take_all || key > prefix);
    const bool eq = cand && !take_all && key == prefix;
    int eq_tot;
    const int eq_rank = eq_seen + block_scan<NT>(eq ? 1 : 0, scan_buf, &eq_tot);
    const bool sel = gt || (eq && eq_rank < remaining);
    int sel_tot;
    const int pos = taken + block_scan<NT>(sel ? 1 : 0, scan_buf, &sel_tot);
    if (sel) {
      a.out_chunks[pos] = i;
      a.out_scores[pos] = a.scores[i];
      if (a.seg_start) {
        a.seg_start[pos] = a.chunk_start[i];
        a.seg_len[pos] = a.chunk_len[i];
      }
    }
    taken += sel_tot;
    eq_seen += eq_tot;
  };
  // in index order, one block-wide step of NT scores at a time
#pragma unroll
  for (int j = 0; j < NR; ++j)
    if (j * NT < a.N) emit(tid + j * NT, kr[j]);
  for (int i0 = NR * NT; i0 < a.N; i0 += NT) {
    const int i = i0 + tid;
    emit(i, i < a.N ? key_of(i) : 0u);
  }
  for (int j = taken + tid; j < a.k; j += NT) {
    a.out_chunks[j] = -1;
    a.out_scores[j] = -INFINITY;
    if (a.seg_start) {
      a.seg_start[j] = 0;
      a.seg_len[j] = 0;
    }
  }
  if (tid == 0) a.out_count[0] = taken;
}

}  // namespace

hipError_t launch_token_mean(const uint16_t* x, int L, int dm, float* out, hipStream_t stream) {
  const int blocks = (dm + kMeanCols - 1) / kMeanCols;
  hipLaunchKernelGGL(token_mean_kernel, dim3(blocks), dim3(kMeanThreads), 0, stream, x, L, dm, out);
  return hipGetLastError();
}

hipError_t launch_chunk_scores(const float* qf, const float* cf, int N, int dm, float* scores, hipStream_t stream) {
  const int waves = N < 4096 ? N : 4096;
  const int blocks = (waves + 3) / 4;
  hipLaunchKernelGGL(chunk_scores_kernel, dim3(blocks), dim3(256), 0, stream, qf, cf, N, dm, scores);
  return hipGetLastError();
}

hipError_t launch_topk(const float* scores, int N, int k, float min_score, const int64_t* chunk_start,
                       const int32_t* chunk_len, int32_t* out_chunks, float* out_scores, int64_t* seg_start,
                       int32_t* seg_len, int32_t* out_count, hipStream_t stream) {
  TopkArgs a{scores, N, k, min_score, chunk_start, chunk_len, out_chunks, out_scores, seg_start, seg_len, out_count};
  if (N <= 256)   // one score per thread (measured: 7.8 vs 9.3 us at N = 256; slower from N = 1000)
    hipLaunchKernelGGL(topk_kernel<256>, dim3(1), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(topk_kernel<kTopkThreads>, dim3(1), dim3(kTopkThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vico
