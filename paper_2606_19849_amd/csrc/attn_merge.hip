// Log-sum-exp merge of attention over split key ranges, for gfx950.
//
// Each part s of a row's key range left a normalised partial output O_s and
// its log2-sum-exp lse_s in the workspace; the whole-range result is
//     lse = log2 sum_s 2^lse_s,   O = sum_s 2^(lse_s - lse) O_s
// (a part that saw no key of the row carries lse_s = -inf and is skipped;
// its O_s slot may never have been written).
//
// Few parts (up to 16, the chunk prefill splits) over many rows: one thread
// per 4 columns of a row loads all parts together.  Many parts (up to 64, short
// queries): a thread walking them one by one is bound by load latency, so a
// work-group of 256 threads takes RPB rows, and for each row PG groups of
// threads take every PG-th part and D/4 threads the 4-float columns -- all
// loads of a row are then in flight together.  The part weights come from
// one wave-wide max and sum over the parts (lane = part).

#include <algorithm>

#include "attn_common.h"

namespace vico {
namespace {

constexpr int kMergeThreads = 256;
constexpr int kFewParts = 16;    // up to here one thread per (row, 4 columns) loads all parts
constexpr int kPartsPerThread = 8;   // many parts: parts one thread loads (64 parts over 8 part groups)

// With an append requested, the blocks past `merge_blocks` copy the chunk's
// K/V into the ring instead of merging: this launch runs after every read of
// the window, so the ring slots it overwrites are free.
__device__ __forceinline__ bool append_block(const AttnArgs& a, int merge_blocks) {
  if ((int)blockIdx.x < merge_blocks) return false;
  const AppendArgs ap{a.kc, a.vc, a.app_rk, a.app_rv, a.C, a.R, a.app_p0, a.Hkv * a.D};
  const int64_t n = (int64_t)(gridDim.x - merge_blocks) * blockDim.x;
  append_units(ap, (int64_t)(blockIdx.x - merge_blocks) * blockDim.x + threadIdx.x, n);
  return true;
}

// Few parts, many rows (chunk prefill splits): one thread per (head, row,
// 4-column group) reads every part's value at once; neighbouring threads
// read neighbouring columns, so every load is a full coalesced row.
template <int D, int NP>
__global__ __launch_bounds__(kMergeThreads) void attn_merge_rows_kernel(AttnArgs a, int merge_blocks) {
  if (append_block(a, merge_blocks)) return;
  constexpr int NQ = D / 4;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n_rows = (int64_t)a.Hq * a.C;
  if (idx >= n_rows * NQ) return;
  const int dq = (int)(idx % NQ);
  const int64_t hr = idx / NQ;
  // every part's lse and O of this thread are loaded together (NP >= the
  // parts, unrolled; the launch takes the smallest of 2, 4, 8, 16 that
  // covers them), so one memory latency covers the whole row.  The O
  // loads do not wait for the lse values: a part past the last reads the last
  // part's slot, and an empty part (lse = -inf, its O slot possibly never
  // written) is dropped by the select in the sum, whatever its slot holds.
  float ls[NP];
  f32x4 os[NP];
#pragma unroll
  for (int s = 0; s < NP; ++s) {
    const int sc = min(s, a.splits - 1);
    ls[s] = s < a.splits ? a.ws_lse[s * n_rows + hr] : -INFINITY;
    os[s] = *(const f32x4*)(a.ws_o + (sc * n_rows + hr) * D + dq * 4);
  }
  float mx = -INFINITY;
#pragma unroll
  for (int s = 0; s < NP; ++s) mx = fmaxf(mx, ls[s]);
  const float m_use = (mx == -INFINITY) ? 0.f : mx;
  f32x4 acc{0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
#pragma unroll
  for (int s = 0; s < NP; ++s) {
    const float w = ls[s] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ls[s] - m_use);
    wsum += w;
    acc += ls[s] == -INFINITY ? f32x4{0.f, 0.f, 0.f, 0.f} : w * os[s];
  }
  acc *= wsum > 0.f ? 1.f / wsum : 0.f;
  const int row = (int)(hr % a.C);
  const int h = (int)(hr / a.C);
  const int64_t oo = ((int64_t)row * a.Hq + h) * D + dq * 4;
  if (a.out_f32) {
    *(f32x4*)((float*)a.out + oo) = acc;
  } else {
    *(bf16x4*)((__bf16*)a.out + oo) = bf16x4{(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
  }
  if (dq == 0 && a.lse) a.lse[(int64_t)h * a.C + row] = wsum > 0.f ? (m_use + __log2f(wsum)) * kLn2 : -INFINITY;
}

// Many parts (short queries): see the file comment.

template <int D>
__global__ __launch_bounds__(kMergeThreads) void attn_merge_kernel(AttnArgs a, int PG, int RPB, int merge_blocks) {
  if (append_block(a, merge_blocks)) return;      // whole blocks: before any barrier
  constexpr int NQ = D / 4;                       // float4 columns per row
  __shared__ float w_s[kMergeThreads / NQ][64];   // per row of the block: part weights
  __shared__ float inv_s[kMergeThreads / NQ];
  __shared__ float lse_s[kMergeThreads / NQ];
  __shared__ f32x4 acc_s[kMergeThreads];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t n_rows = (int64_t)a.Hq * a.C;
  const int64_t stride = n_rows;                  // parts are [splits][Hq][C]
  const int64_t r0 = (int64_t)blockIdx.x * RPB;

  // weights of every row of the block: wave w takes rows w, w+4, ...
  for (int r = wave; r < RPB; r += kMergeThreads / 64) {
    const int64_t hr = r0 + r;
    float ls = -INFINITY;
    if (hr < n_rows && lane < a.splits) ls = a.ws_lse[lane * stride + hr];
    float mx = ls;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    const float m_use = (mx == -INFINITY) ? 0.f : mx;
    const float w = (ls == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ls - m_use);
    float sum = w;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o, 64);
    w_s[r][lane] = w;
    if (lane == 0) {
      inv_s[r] = sum > 0.f ? 1.f / sum : 0.f;
      lse_s[r] = sum > 0.f ? (m_use + __log2f(sum)) * kLn2 : -INFINITY;
    }
  }
  __syncthreads();

  // thread = (row r, part group pg, column dq)
  const int dq = tid % NQ;
  const int pg = (tid / NQ) % PG;
  const int r = tid / (NQ * PG);
  const int64_t hr = r0 + r;
  f32x4 acc{0.f, 0.f, 0.f, 0.f};
  if (r < RPB && hr < n_rows) {
    // this thread's parts pg, pg + PG, ... (at most kPartsPerThread): every
    // load is issued before the first is used, so the row costs one memory
    // latency; the sum runs over the parts in the same order as a plain loop
    float w[kPartsPerThread];
    f32x4 v[kPartsPerThread];
#pragma unroll
    for (int i = 0; i < kPartsPerThread; ++i) {
      // unconditional loads (a part past the last, or one that saw no key and
      // left its slot unwritten, reads a slot in range and gets weight 0; the
      // select below drops whatever it holds)
      const int p = pg + i * PG;
      const int pc = min(p, a.splits - 1);
      w[i] = p < a.splits ? w_s[r][p] : 0.f;
      v[i] = *(const f32x4*)(a.ws_o + (pc * stride + hr) * D + dq * 4);
    }
#pragma unroll
    for (int i = 0; i < kPartsPerThread; ++i)
      if (pg + i * PG < a.splits) acc += w[i] != 0.f ? w[i] * v[i] : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  acc_s[tid] = acc;
  __syncthreads();
  if (pg != 0 || r >= RPB || hr >= n_rows) return;
  for (int g = 1; g < PG; ++g) acc += acc_s[tid + g * NQ];
  acc *= inv_s[r];
  const int row = (int)(hr % a.C);
  const int h = (int)(hr / a.C);
  const int64_t oo = ((int64_t)row * a.Hq + h) * D + dq * 4;
  if (a.out_f32) {
    *(f32x4*)((float*)a.out + oo) = acc;
  } else {
    *(bf16x4*)((__bf16*)a.out + oo) = bf16x4{(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
  }
  if (dq == 0 && a.lse) a.lse[(int64_t)h * a.C + row] = lse_s[r];
}

}  // namespace

hipError_t launch_merge(const AttnArgs& a, hipStream_t stream) {
  if (a.splits < 1 || a.splits > 64) return hipErrorInvalidValue;   // one wave holds the part weights
  const int64_t rows = (int64_t)a.Hq * a.C;
  // copy blocks for the append (one 16-byte unit per thread per step)
  const int64_t app_units = a.app_rk ? 2 * (int64_t)a.C * (a.Hkv * a.D / 8) : 0;
  const int app_blocks = (int)std::min<int64_t>((app_units + kMergeThreads - 1) / kMergeThreads, 2048);
  if (a.splits <= kFewParts) {
    const int blocks = (int)((rows * (a.D / 4) + kMergeThreads - 1) / kMergeThreads);
    const dim3 grid(blocks + app_blocks), block(kMergeThreads);
    if (a.splits <= 2) {
      if (a.D == 128) hipLaunchKernelGGL((attn_merge_rows_kernel<128, 2>), grid, block, 0, stream, a, blocks);
      else hipLaunchKernelGGL((attn_merge_rows_kernel<64, 2>), grid, block, 0, stream, a, blocks);
    } else if (a.splits <= 4) {
      if (a.D == 128) hipLaunchKernelGGL((attn_merge_rows_kernel<128, 4>), grid, block, 0, stream, a, blocks);
      else hipLaunchKernelGGL((attn_merge_rows_kernel<64, 4>), grid, block, 0, stream, a, blocks);
    } else if (a.splits <= 8) {
      if (a.D == 128) hipLaunchKernelGGL((attn_merge_rows_kernel<128, 8>), grid, block, 0, stream, a, blocks);
      else hipLaunchKernelGGL((attn_merge_rows_kernel<64, 8>), grid, block, 0, stream, a, blocks);
    } else {
      if (a.D == 128) hipLaunchKernelGGL((attn_merge_rows_kernel<128, 16>), grid, block, 0, stream, a, blocks);
      else hipLaunchKernelGGL((attn_merge_rows_kernel<64, 16>), grid, block, 0, stream, a, blocks);
    }
    return hipGetLastError();
  }
  // part groups: the parts rounded up to a power of two, at most what one row's
  // columns leave of the 256 threads; the remaining threads take more rows
  const int nq = a.D / 4;
  int pg = 1;
  while (pg < a.splits && pg * 2 * nq <= kMergeThreads) pg *= 2;
  if (pg * kPartsPerThread < a.splits) return hipErrorInvalidValue;
  const int rpb = kMergeThreads / (nq * pg);
  const int blocks = (int)((rows + rpb - 1) / rpb);
  if (a.D == 128)
    hipLaunchKernelGGL(attn_merge_kernel<128>, dim3(blocks + app_blocks), dim3(kMergeThreads), 0, stream, a, pg, rpb,
                       blocks);
  else
    hipLaunchKernelGGL(attn_merge_kernel<64>, dim3(blocks + app_blocks), dim3(kMergeThreads), 0, stream, a, pg, rpb,
                       blocks);
  return hipGetLastError();
}

}  // namespace vico
