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
//     rounded to bf16, are already the B operand (k index = key slot, keys
//     of each 16-key group in the order the accumulator produces them); the
//     A operand V^T is read from the row-major V tile with the gfx950
//     transposing LDS read ds_read_b64_tr_b16 (each 16-lane group reads a
//     4-key x 16-dim block and lane i receives dim i of the 4 keys).  O^T stays
//     in the layout "lane = query row", so per-row rescale factors are
//     lane-local.
//   * Online softmax in fp32 with exp2 (v_exp_f32), scale*log2(e) folded into
//     one FMA per logit.  The running max is only raised (and O rescaled)
//     when some row's tile max exceeds it by more than 2^8; until then the
//     probabilities are exp2 of at most 8, exact in fp32 and bf16 range.
//   * K/V tiles: 8192/d keys, double-buffered in LDS; the next tile's loads
//     are in flight while the current tile is multiplied.  Loads go through
//     buffer resources (one per sink / ring / chunk tensor): a tile that lies
//     inside one segment (and does not cross the ring end) is addressed as a
//     scalar tile base plus a fixed per-thread offset; the few tiles that
//     straddle a boundary resolve each key row (ring slot = ws + k, minus R
//     once past the end) and read all three resources with out-of-range
//     offsets for the wrong ones, which the hardware returns as zero.  Keys
//     past the chunk end read as zero the same way.  No copies are made.
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
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __amdgpu_buffer_rsrc_t rsrc_t;

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

// Raw buffer resource over `bytes` bytes (stride 0, 32-bit data format).
// Reads at offsets >= bytes return zero.
__device__ __forceinline__ rsrc_t make_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr float kRescaleThreshold = 8.0f;   // log2 units

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(AttnArgs a, int n_rt, int g) {
  constexpr int BN = 8192 / D;     // keys per tile
  constexpr int NB = BN / 32;      // 32-key blocks of S^T per tile
  constexpr int NKS = D / 16;      // k-steps of Q K^T
  constexpr int NDB = D / 32;      // 32-dim blocks of O^T
  constexpr int NPK = BN / 16;     // 16-key k-steps of V^T P^T
  constexpr int NCH = D / 8;       // 16-byte chunks per key row
  // LDS row strides (elements).  The LDS has 64 banks of 4 bytes.  K rows are
  // read 16 lanes x 16 bytes at a time from 16 consecutive rows: a stride of
  // 4 banks mod 64 (16 B pad) keeps them apart.  V rows are read by the
  // transposing loads 32 lanes at a time as 4 rows x 64 bytes: a stride of
  // 64 bytes mod 256 puts the 4 rows on disjoint banks (d = 128).
  constexpr int KSTR = D + 8;
  constexpr int VSTR = D == 128 ? D + 32 : D + 8;
  constexpr int KT = BN * KSTR;    // elements of one K tile
  constexpr int VT = BN * VSTR;    // elements of one V tile
  static_assert((BN / 4) * NCH == kThreads, "one 4-key x 8-dim block per thread");

  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (KT + VT)];   // {K, V} x 2 buffers

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
  const int rb = a.Hkv * D * 2;                                // bytes per token row
  const uint32_t colb = (uint32_t)(kv * D + dc * 8) * 2u;      // byte offset inside a row
  const uint32_t thr_off = (uint32_t)(kg * 4) * (uint32_t)rb + colb;
  const rsrc_t rs_sk = make_rsrc(a.sink_k, S * rb), rs_sv = make_rsrc(a.sink_v, S * rb);
  const rsrc_t rs_rk = make_rsrc(a.ring_k, a.R * rb), rs_rv = make_rsrc(a.ring_v, a.R * rb);
  const rsrc_t rs_ck = make_rsrc(a.kc, C * rb), rs_cv = make_rsrc(a.vc, C * rb);

  u32x4 kr[4], vr[4];
  auto load_tile = [&](int t) {
    const int k0 = t * BN, k1 = k0 + BN;
    // segment of the whole tile (wave-uniform): 0 sink, 1 ring without wrap, 2 chunk, 3 mixed
    int mode = 3, row_base = 0;
    if (k1 <= S) {
      mode = 0; row_base = k0;
    } else if (k0 >= SW) {
      mode = 2; row_base = k0 - SW;
    } else if (k0 >= S && k1 <= SW) {
      int slot0 = a.ws + (k0 - S);
      if (slot0 >= a.R) slot0 -= a.R;
      if (slot0 + BN <= a.R) { mode = 1; row_base = slot0; }
    }
    if (mode != 3) {
      // select scalar base and size, then build one resource (keeps it in SGPRs)
      const uint16_t* bk = mode == 0 ? a.sink_k : (mode == 1 ? a.ring_k : a.kc);
      const uint16_t* bv = mode == 0 ? a.sink_v : (mode == 1 ? a.ring_v : a.vc);
      const int nb = mode == 0 ? S * rb : (mode == 1 ? a.R * rb : C * rb);
      const rsrc_t rk_ = make_rsrc(bk, nb), rv_ = make_rsrc(bv, nb);
      const uint32_t off = (uint32_t)row_base * (uint32_t)rb + thr_off;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        kr[r] = __builtin_amdgcn_raw_buffer_load_b128(rk_, off + r * rb, 0, 0);
        vr[r] = __builtin_amdgcn_raw_buffer_load_b128(rv_, off + r * rb, 0, 0);
      }
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kk = k0 + kg * 4 + r;
        int slot = a.ws + (kk - S);
        if (slot >= a.R) slot -= a.R;
        const uint32_t o_s = kk < S ? (uint32_t)kk * rb + colb : kOutOfRange;
        const uint32_t o_r = (kk >= S && kk < SW) ? (uint32_t)slot * rb + colb : kOutOfRange;
        const uint32_t o_c = kk >= SW ? (uint32_t)(kk - SW) * rb + colb : kOutOfRange;
        kr[r] = __builtin_amdgcn_raw_buffer_load_b128(rs_sk, o_s, 0, 0) |
                __builtin_amdgcn_raw_buffer_load_b128(rs_rk, o_r, 0, 0) |
                __builtin_amdgcn_raw_buffer_load_b128(rs_ck, o_c, 0, 0);
        vr[r] = __builtin_amdgcn_raw_buffer_load_b128(rs_sv, o_s, 0, 0) |
                __builtin_amdgcn_raw_buffer_load_b128(rs_rv, o_r, 0, 0) |
                __builtin_amdgcn_raw_buffer_load_b128(rs_cv, o_c, 0, 0);
      }
    }
  };

  auto store_tile = [&](int buf) {
    uint16_t* Ks = smem + buf * (KT + VT);
    uint16_t* Vs = Ks + KT;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      *(u32x4*)(Ks + (kg * 4 + r) * KSTR + dc * 8) = kr[r];
      *(u32x4*)(Vs + (kg * 4 + r) * VSTR + dc * 8) = vr[r];
    }
  };

  // Per-lane source of the transposing V reads: 16-lane group G = lane/16
  // covers dims (G%2)*16 .. +15 of a 32-dim block and k-slots (G/2)*8 ..;
  // its lane 4j+q supplies key j of the group's 4 keys, dims 4q .. 4q+3.
  const int v_lane_off = ((lane >> 5) * 4 + ((lane & 15) >> 2)) * VSTR + ((lane >> 4) & 1) * 16 + (lane & 3) * 4;

  // ---- running state of this lane's row (both halves hold the same m)
  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x16{};
  float m_run = -INFINITY;
  float l_run = 0.f;
  const float c = a.scale_log2;

  auto compute_tile = [&](int buf, int k0) {
    const uint16_t* Ks = smem + buf * (KT + VT);
    const uint16_t* Vs = Ks + KT;
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
    mx = pair_max(mx) * c;
    if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescaleThreshold)) {
      const float m_new = fmaxf(m_run, mx);
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
    const uint16_t* vl = Vs + v_lane_off;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
#pragma unroll
      for (int kp = 0; kp < NPK; ++kp) {
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vl + (kp * 16) * VSTR + db * 32));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vl + (kp * 16 + 8) * VSTR + db * 32));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
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
