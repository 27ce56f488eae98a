// Bounded chunk-prefill attention for gfx950 (CDNA4).
//
// Computes softmax(Q K^T / sqrt(d)) V for the rows of one visual chunk over
// the keys [sink | W newest history tokens (read through ring slots) |
// chunk keys 0..i] -- the bounded visual attention of ViCoStream (Sec. 3,
// "LLM Prefilling and Decoding"; visibility as in the vision rows of Eq. (4),
// at token granularity, causal inside the chunk).
//
// Mapping onto the hardware
//   * Work-group = 4 waves = 128 query rows of one query head (one key range
//     when split).  Each wave owns 32 rows for the whole key loop.
//   * S^T = K Q^T with v_mfma_f32_32x32x16_bf16: the K tile (from LDS) is the
//     A operand, the wave's Q rows (held in VGPRs for the whole loop) the B
//     operand.  In the accumulator layout lane l then holds 16 logits of
//     query row l%32, and lanes l and l+32 together hold all 32 keys of the
//     block, so the row max / row sum need a single v_permlane32_swap.
//   * O^T = V^T P^T with the same MFMA: the S^T accumulator registers,
//     rounded to bf16, are already the B operand (k index = key slot); the A
//     operand is V^T, which the loader writes into LDS transposed, with the
//     keys of each 16-key group permuted to the order the accumulator layout
//     produces them in.  O^T stays in the layout "lane = query row", so the
//     per-row rescale factors are lane-local.
//   * Online softmax in fp32 with exp2 (v_exp_f32), scale*log2(e) folded into
//     one FMA per logit.
//   * K/V tiles: 8192/d keys, double-buffered in LDS; the next tile's global
//     loads are in flight while the current tile is multiplied.  The window
//     start and the ring wrap are resolved per key row when loading: slot =
//     ws + k, minus R once if it passed the end.  No copies are made.
//   * Causal chunk: only tiles that reach past the first row of a wave are
//     masked; tiles beyond the last row of a wave are skipped by that wave.
//   * Work-groups are renumbered so that consecutive logical ids (the query
//     heads of one KV head) land on the same XCD and share its L2.
//   * Optional split of the key range (for chunks too small to fill 256 CUs):
//     each split writes fp32 O and log2-sum-exp; a merge kernel combines them.

#include "vico_internal.h"

namespace vico {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLn2 = 0.6931471805599453f;
constexpr int kNumXcd = 8;

// Logical work-group id for physical id `pid` so that each XCD receives a
// contiguous block of logical ids (hardware dispatches ids round-robin over
// the XCDs).  A bijection on [0, n).
__device__ __forceinline__ int xcd_remap(int pid, int n) {
  const int xcd = pid % kNumXcd, local = pid / kNumXcd;
  const int per = n / kNumXcd, rem = n % kNumXcd;
  return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// Combine lane l with lane l^32 (the two halves of one query row's keys).
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// XOR swizzle of 16-byte segments in the V^T tile rows: spreads both the
// transposing writes (rows 8 apart) and the MFMA operand reads (8
// consecutive rows) over distinct LDS banks.
__device__ __forceinline__ int vswz(int d) { return (d ^ (d >> 3)) & 7; }

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(AttnArgs a, int n_rt, int g) {
  constexpr int BN = 8192 / D;     // keys per tile
  constexpr int NB = BN / 32;      // 32-key blocks of S^T per tile
  constexpr int NKS = D / 16;      // k-steps of Q K^T
  constexpr int NDB = D / 32;      // 32-dim blocks of O^T
  constexpr int NPK = BN / 16;     // 16-key k-steps of V^T P^T
  constexpr int NCH = D / 8;       // 16-byte chunks per key row
  constexpr int KSTR = D + 8;      // K tile row stride in elements (16 B pad)
  constexpr int VROW = BN;         // V^T tile row length in elements
  constexpr int KT = BN * KSTR;
  constexpr int VT = D * VROW;
  static_assert((BN / 4) * NCH == kThreads, "one 4-key x 8-dim block per thread");

  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (KT + VT)];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int hh = lane >> 5;

  // ---- which rows / head / key range this work-group owns
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int qh = L % g;
  int rest = L / g;
  const int rt = n_rt - 1 - rest % n_rt;   // longest row tiles first
  rest /= n_rt;
  const int sp = rest % a.splits;
  const int kv = rest / a.splits;
  const int h = kv * g + qh;

  const int C = a.C, S = a.S, SW = a.S + a.Wv;
  const int row0 = rt * kBlockM;
  const int row_last = min(row0 + kBlockM, C) - 1;
  const int n_tiles = (SW + row_last + 1 + BN - 1) / BN;
  const int t_lo = (int)((int64_t)n_tiles * sp / a.splits);
  const int t_hi = (int)((int64_t)n_tiles * (sp + 1) / a.splits);

  const int wrow0 = row0 + wave * 32;
  const int row = wrow0 + l32;
  const bool wave_active = wrow0 < C;
  const int row_c = min(row, C - 1);
  const int key_lim = SW + row_c;                       // last key visible to this row
  const int wave_first_lim = SW + min(wrow0, C - 1);    // ... to the wave's first row
  const int wave_last_lim = SW + min(wrow0 + 31, C - 1);

  // ---- Q rows of this wave as MFMA B fragments (lane: row l32, dims hh*8..+8)
  bf16x8 qf[NKS];
  {
    const uint16_t* qp = a.q + ((int64_t)row_c * a.Hq + h) * D + hh * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      u32x4 v = (row < C) ? *(const u32x4*)(qp + ks * 16) : u32x4{0u, 0u, 0u, 0u};
      qf[ks] = __builtin_bit_cast(bf16x8, v);
    }
  }

  // ---- tile loader: thread = 4 consecutive keys x one 16-byte dim chunk
  const int kg = tid / NCH;
  const int dc = tid % NCH;
  const int64_t kvs = (int64_t)a.Hkv * D;
  const int64_t col = (int64_t)kv * D + dc * 8;

  u32x4 kr[4], vr[4];
  auto load_tile = [&](int t) {
    const int kbase = t * BN + kg * 4;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int kk = kbase + r;
      const uint16_t* pk = nullptr;
      const uint16_t* pv = nullptr;
      int64_t off = 0;
      if (kk < S) {
        pk = a.sink_k; pv = a.sink_v; off = kk;
      } else if (kk < SW) {
        int slot = a.ws + (kk - S);
        if (slot >= a.R) slot -= a.R;
        pk = a.ring_k; pv = a.ring_v; off = slot;
      } else if (kk < SW + C) {
        pk = a.kc; pv = a.vc; off = kk - SW;
      }
      if (pk) {
        kr[r] = *(const u32x4*)(pk + off * kvs + col);
        vr[r] = *(const u32x4*)(pv + off * kvs + col);
      } else {
        kr[r] = u32x4{0u, 0u, 0u, 0u};
        vr[r] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };

  // V^T slot of key 4*kg within the tile: inside each 16-key group the keys
  // are stored in the order the S^T accumulator hands them to lane halves.
  const int vgrp = kg >> 2, va = kg & 3;
  const int vslot = vgrp * 16 + (va & 1) * 8 + (va >> 1) * 4;
  const int vseg = vslot >> 3, vhalf = (vslot >> 2) & 1;

  auto store_tile = [&](int buf) {
    uint16_t* Ks = smem + buf * (KT + VT);
    uint16_t* Vt = Ks + KT;
#pragma unroll
    for (int r = 0; r < 4; ++r) *(u32x4*)(Ks + (kg * 4 + r) * KSTR + dc * 8) = kr[r];
#pragma unroll
    for (int m = 0; m < 4; ++m) {      // dword m of a row holds dims 2m (low) and 2m+1 (high)
      u32x2 lo, hi;
      lo[0] = __builtin_amdgcn_perm(vr[1][m], vr[0][m], 0x05040100u);
      lo[1] = __builtin_amdgcn_perm(vr[3][m], vr[2][m], 0x05040100u);
      hi[0] = __builtin_amdgcn_perm(vr[1][m], vr[0][m], 0x07060302u);
      hi[1] = __builtin_amdgcn_perm(vr[3][m], vr[2][m], 0x07060302u);
      const int d0 = dc * 8 + 2 * m, d1 = d0 + 1;
      *(u32x2*)(Vt + d0 * VROW + ((vseg ^ vswz(d0)) << 3) + vhalf * 4) = lo;
      *(u32x2*)(Vt + d1 * VROW + ((vseg ^ vswz(d1)) << 3) + vhalf * 4) = hi;
    }
  };

  // ---- running state of this lane's row (both halves hold the same m)
  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x16{};
  float m_run = -INFINITY;
  float l_run = 0.f;
  const float c = a.scale_log2;

  auto compute_tile = [&](int buf, int k0) {
    const uint16_t* Ks = smem + buf * (KT + VT);
    const uint16_t* Vt = Ks + KT;
    f32x16 s[NB];
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) {
      s[kb] = f32x16{};
      const uint16_t* kp = Ks + (kb * 32 + l32) * KSTR + hh * 8;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const bf16x8 kf = *(const bf16x8*)(kp + ks * 16);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[kb], 0, 0, 0);
      }
    }
    if (k0 + BN - 1 > wave_first_lim) {     // tile reaches into the causal part for this wave
#pragma unroll
      for (int kb = 0; kb < NB; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int kk = k0 + kb * 32 + 8 * (v >> 2) + hh * 4 + (v & 3);
          if (kk > key_lim) s[kb][v] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NB; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kb][v]);
    mx = pair_max(mx);
    const float m_new = fmaxf(m_run, mx * c);
    if (__builtin_amdgcn_ballot_w64(m_new > m_run)) {
      const float alpha = (m_new == m_run) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= alpha;
      m_run = m_new;
    }
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
    float lsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < NB; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][v], c, -m_use));
        s[kb][v] = p;
        lsum += p;
      }
    l_run += lsum;
    bf16x8 pf[NPK];
#pragma unroll
    for (int kp = 0; kp < NPK; ++kp)
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[kp][e] = (__bf16)s[kp >> 1][(kp & 1) * 8 + e];
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int d = db * 32 + l32;
      const uint16_t* vrow = Vt + d * VROW;
      const int sw = vswz(d);
#pragma unroll
      for (int kp = 0; kp < NPK; ++kp) {
        const bf16x8 vf = *(const bf16x8*)(vrow + (((kp * 2 + hh) ^ sw) << 3));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kp], o[db], 0, 0, 0);
      }
    }
  };

  // ---- key loop: one barrier per tile, next tile's loads in flight
  if (t_lo < t_hi) {
    load_tile(t_lo);
    store_tile(0);
    __syncthreads();
    for (int t = t_lo; t < t_hi; ++t) {
      const int buf = (t - t_lo) & 1;
      const bool more = t + 1 < t_hi;
      if (more) load_tile(t + 1);
      const int k0 = t * BN;
      if (wave_active && k0 <= wave_last_lim) compute_tile(buf, k0);
      if (more) store_tile(buf ^ 1);
      __syncthreads();
    }
  }

  if (!wave_active) return;
  const float l_tot = pair_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse2 = l_tot > 0.f ? m_run + __log2f(l_tot) : -INFINITY;
  if (row >= C) return;

  if (a.splits == 1) {
    if (a.out_f32) {
      float* op = (float*)a.out + ((int64_t)row * a.Hq + h) * D + hh * 4;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          f32x4 v{o[db][q4 * 4] * inv, o[db][q4 * 4 + 1] * inv, o[db][q4 * 4 + 2] * inv, o[db][q4 * 4 + 3] * inv};
          *(f32x4*)(op + db * 32 + q4 * 8) = v;
        }
    } else {
      __bf16* op = (__bf16*)a.out + ((int64_t)row * a.Hq + h) * D + hh * 4;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          bf16x4 v{(__bf16)(o[db][q4 * 4] * inv), (__bf16)(o[db][q4 * 4 + 1] * inv),
                   (__bf16)(o[db][q4 * 4 + 2] * inv), (__bf16)(o[db][q4 * 4 + 3] * inv)};
          *(bf16x4*)(op + db * 32 + q4 * 8) = v;
        }
    }
    if (a.lse && hh == 0) a.lse[(int64_t)h * C + row] = lse2 * kLn2;
  } else {
    float* op = a.ws_o + (((int64_t)sp * a.Hq + h) * C + row) * D + hh * 4;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        f32x4 v{o[db][q4 * 4] * inv, o[db][q4 * 4 + 1] * inv, o[db][q4 * 4 + 2] * inv, o[db][q4 * 4 + 3] * inv};
        *(f32x4*)(op + db * 32 + q4 * 8) = v;
      }
    if (hh == 0) a.ws_lse[((int64_t)sp * a.Hq + h) * C + row] = lse2;
  }
}

// Merge of split key ranges: O = sum_s 2^(lse_s - lse) O_s, lse = log2 sum_s 2^lse_s.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int NQ = D / 4;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)a.Hq * a.C * NQ;
  if (idx >= total) return;
  const int dq = (int)(idx % NQ);
  const int64_t hr = idx / NQ;
  const int row = (int)(hr % a.C);
  const int h = (int)(hr / a.C);
  const int64_t stride_s = (int64_t)a.Hq * a.C;
  float mx = -INFINITY;
  for (int s = 0; s < a.splits; ++s) mx = fmaxf(mx, a.ws_lse[s * stride_s + hr]);
  const float m_use = (mx == -INFINITY) ? 0.f : mx;
  f32x4 acc{0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
  for (int s = 0; s < a.splits; ++s) {
    const float w = __builtin_amdgcn_exp2f(a.ws_lse[s * stride_s + hr] - m_use);
    const f32x4 v = *(const f32x4*)(a.ws_o + (s * stride_s + hr) * D + dq * 4);
    wsum += w;
    acc += w * v;
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  acc *= inv;
  const int64_t oo = ((int64_t)row * a.Hq + h) * D + dq * 4;
  if (a.out_f32) {
    *(f32x4*)((float*)a.out + oo) = acc;
  } else {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    *(bf16x4*)((__bf16*)a.out + oo) = bf16x4{(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
  }
  if (dq == 0 && a.lse) a.lse[(int64_t)h * a.C + row] = wsum > 0.f ? (m_use + __log2f(wsum)) * kLn2 : -INFINITY;
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream) {
  const int g = a.Hq / a.Hkv;
  const int n_rt = (a.C + kBlockM - 1) / kBlockM;
  const int nwg = a.Hq * n_rt * a.splits;
  if (a.D == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3(nwg), dim3(kThreads), 0, stream, a, n_rt, g);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3(nwg), dim3(kThreads), 0, stream, a, n_rt, g);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || a.splits == 1) return err;
  const int64_t total = (int64_t)a.Hq * a.C * (a.D / 4);
  const int blocks = (int)((total + 255) / 256);
  if (a.D == 128)
    hipLaunchKernelGGL(attn_merge_kernel<128>, dim3(blocks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_merge_kernel<64>, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vico
