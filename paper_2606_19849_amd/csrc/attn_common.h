// Device helpers shared by the attention kernels of libvico (gfx950 only).
#pragma once

#include "vico_internal.h"

namespace vico {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr float kLn2 = 0.6931471805599453f;
constexpr int kNumXcd = 8;
constexpr uint32_t kOutOfRange = 0x80000000u;
// Largest lane sum of one half's 16 probabilities accepted against the
// running max; it bounds each of them by 2^8 (exp2 of at most 8), far inside
// the fp32 and bf16 range.
constexpr float kLaneSumLimit = 256.0f;

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

// 16 bytes per lane from a buffer straight into LDS: lane i writes lds + 16*i.
// Kept in a device-only function: used inline in a kernel body, the builtin
// makes the host compilation pass drop the kernel's launch stub.
__device__ __forceinline__ void load_lds16(rsrc_t r, lds_void* lds, uint32_t voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, voffset, 0, 0, 0);
}

// s_waitcnt immediate: vmcnt(n), lgkmcnt(0), expcnt not waited for.
constexpr uint32_t waitcnt_vm_lgkm0(uint32_t n) { return 0x0070u | n; }

// ---------------------------------------------------------------------------
// The attention tile body shared by the chunk-prefill and gathered-query
// kernels: one wave's 32 query rows against 64-key K/V tiles held in LDS
// (the attention of Sec. 3, "LLM Prefilling and Decoding", computed with an
// online softmax).
//
//   * S^T = K Q^T with v_mfma_f32_32x32x16_bf16: a K fragment read from LDS is
//     the A operand, the wave's Q rows (VGPRs, whole loop) the B operand.  In
//     the accumulator layout lane l holds 16 logits of query row l%32; lanes
//     l and l+32 together hold the 32 keys of a half tile, so a row reduction
//     takes one v_permlane32_swap.
//   * O^T = V^T P^T with the same MFMA: the S^T accumulator rounded to bf16
//     is already the B operand (k index = key slot in the order the
//     accumulator produces them); the A operand V^T comes from the row-major
//     V tile through the transposing read ds_read_b64_tr_b16 (each 16-lane
//     group reads a 4-key x 16-dim block; lane i receives dim i of the 4
//     keys).  O^T keeps "lane = query row", so per-row factors are lane-local.
//   * Softmax in fp32 with exp2, scale*log2(e) folded into one FMA per logit.
//     Each half is exponentiated against the running max straight away; the
//     max is raised (O and l rescaled, the half redone) only when some lane's
//     sum of probabilities exceeds 2^8, which bounds every probability by
//     2^8, or while a row has no max yet.  No row-max reduction sits between
//     the logits and the exponentials.
//
// LDS tiles are dense rows of 2*D bytes with 16-byte units permuted inside a
// row against bank conflicts (64 banks of 4 bytes):
//   K: unit u of row r at u ^ lds_swz_k(r): a K fragment read serves 16 lanes
//      = 16 consecutive rows at one unit, which the swizzle makes distinct.
//   V: unit u of row r at u ^ lds_swz_v(r): a transposing read serves 32
//      lanes = 4 consecutive rows x 4 units, which the swizzle spreads apart.
template <int D>
__device__ __forceinline__ int lds_swz_k(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
template <int D>
__device__ __forceinline__ int lds_swz_v(int r) { return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1); }

template <int D>
struct WaveTile {
  static constexpr int NKS = D / 16;   // k-steps of Q K^T
  static constexpr int NDB = D / 32;   // 32-dim blocks of O^T
  static constexpr int RBY = D * 2;    // bytes per LDS row

  // The wave's state lives in the kernel (locals, all in VGPRs); the tile
  // body works on it through references, as a closure would.
  const bf16x8 (&qf)[NKS];       // Q rows (lane: row l%32, dims 8*(l/32) + 16*ks .. +8)
  const uint32_t (&k_rd)[NKS];   // per-lane LDS byte offsets of the K fragments
  const uint32_t (&v_rd)[NDB];   //   and of the V^T fragments
  f32x16 (&o)[NDB];              // O^T accumulators
  float& m_run;                  // running max (log2 units) of this lane's row
  float& l_run;                  // this lane's sum of probabilities
  float& neg_m;                  // -m_run, or 0 while m_run is -inf
  const float c;                 // softmax scale * log2(e)

  // Loads this lane's Q row (bf16, 16-byte aligned, at dims 8*(lane/32)) as
  // MFMA B fragments.
  __device__ __forceinline__ static void load_q(bf16x8 (&q)[NKS], const uint16_t* qp) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) q[ks] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qp + ks * 16));
  }

  // Per-lane LDS byte offsets of the operand reads and an empty running state.
  __device__ __forceinline__ static void start(uint32_t (&krd)[NKS], uint32_t (&vrd)[NDB], f32x16 (&acc)[NDB],
                                               float& m, float& l, float& nm) {
    const int lane = threadIdx.x & 63, l32 = lane & 31, hh = lane >> 5;
    //   K fragment (half h, ks): row h*32 + l32, logical unit 2*ks + hh
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) krd[ks] = (uint32_t)(l32 * RBY + (((2 * ks) | hh) ^ lds_swz_k<D>(l32)) * 16);
    //   V^T fragment (db, kp, half): 16-lane group G = lane/16 covers dims
    //   (G%2)*16 .. +15 of a 32-dim block and k-slots (G/2)*8 ..; its lane
    //   4j+q supplies key j of the group's 4 keys (row kp*16 + half*8 +
    //   (G/2)*4 + j), dims 4q .. 4q+3.
    const int j = (lane & 15) >> 2, q = lane & 3;
    const int r = (lane >> 5) * 4 + j;   // row within the 8-row half-group (the swizzle depends on r mod 4 only)
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int u = db * 4 + ((lane >> 4) & 1) * 2 + (q >> 1);
      vrd[db] = (uint32_t)(r * RBY + (u ^ lds_swz_v<D>(r)) * 16 + (q & 1) * 8);
    }
#pragma unroll
    for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};
    m = -INFINITY;
    l = 0.f;
    nm = 0.f;
  }

  // Q K^T for one 32-key half of the tile
  __device__ __forceinline__ void qk_half(const uint16_t* Ks, int h, f32x16& s) const {
    s = f32x16{};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const bf16x8 kf = *(const bf16x8*)((const char*)Ks + h * 32 * RBY + k_rd[ks]);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s, 0, 0, 0);
    }
  }

  // Causal mask of one half: accumulator element v of lane l holds key
  // k0h + 8*(v/4) + 4*(l/32) + v%4; it is dropped when past `key_lim`, the
  // last key visible to the lane's row.
  __device__ __forceinline__ static void mask_half(int k0h, int key_lim, int hh, f32x16& s) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int kk = k0h + 8 * (v >> 2) + hh * 4 + (v & 3);
      if (kk > key_lim) s[v] = -INFINITY;
    }
  }

  // Softmax of one half.  The probabilities are taken against the running
  // max first (exp2, bf16 pack, lane sums).  While no lane sum exceeds 2^8 (a
  // lane's sum bounds each of its 16 terms) that max stays; otherwise, and
  // while the row has no max yet, the max is raised to the half's row max, O
  // and l are rescaled and the half is exponentiated again (rare,
  // wave-uniform branch).
  __device__ __forceinline__ void softmax_half(const f32x16& s, bf16x8 (&pf)[2]) {
    auto expo = [&]() __attribute__((always_inline)) {
      float e[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) e[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c, neg_m));
      float s0 = e[0], s1 = e[1];    // two chains
#pragma unroll
      for (int v = 1; v < 8; ++v) {
        s0 += e[2 * v];
        s1 += e[2 * v + 1];
      }
#pragma unroll
      for (int kp = 0; kp < 2; ++kp)
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) pf[kp][jj] = (__bf16)e[kp * 8 + jj];
      return s0 + s1;
    };
    float lsum = expo();
    if (__builtin_amdgcn_ballot_w64(!(lsum <= kLaneSumLimit) || m_run == -INFINITY)) {
      float mx = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[v]);
      // branch-free per lane: a divergent branch here would keep two copies of O
      const float m_new = fmaxf(m_run, pair_max(mx) * c);
      const float alpha = (m_new == m_run) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= alpha;
      m_run = m_new;
      neg_m = (m_new == -INFINITY) ? 0.f : -m_new;
      lsum = expo();
    }
    l_run += lsum;
  }

  // O^T += V^T P^T for one half
  __device__ __forceinline__ void pv_half(const uint16_t* Vs, int h, const bf16x8 (&pf)[2]) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        const char* vp = (const char*)Vs + v_rd[db] + (h * 32 + kp * 16) * RBY;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)vp);
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vp + 8 * RBY));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kp], o[db], 0, 0, 0);
      }
  }

  // One 64-key tile (key index k0 at LDS row 0) in two 32-key halves, ordered
  // so that the matrix cores multiply one half while the VALU exponentiates
  // the other:  QK(0) | [QK(1) with softmax(0)] [PV(0) with softmax(1)] | PV(1).
  // The wave raises its issue priority while it feeds the matrix cores, so of
  // the two waves sharing a SIMD the one with MFMAs ready goes first and the
  // other's softmax fills the MFMA shadow.  MASK: the causal mask applies
  // (keys past `key_lim` are dropped; hh = lane / 32).
  template <bool MASK>
  __device__ __forceinline__ void tile(const uint16_t* Ks, const uint16_t* Vs, int k0, int key_lim, int hh) {
    f32x16 s0, s1;
    bf16x8 p0[2], p1[2];
    __builtin_amdgcn_s_setprio(1);
    qk_half(Ks, 0, s0);
    __builtin_amdgcn_s_setprio(0);
    if constexpr (MASK) mask_half(k0, key_lim, hh, s0);
    __builtin_amdgcn_s_setprio(1);
    qk_half(Ks, 1, s1);
    softmax_half(s0, p0);
    pv_half(Vs, 0, p0);
    if constexpr (MASK) mask_half(k0 + 32, key_lim, hh, s1);
    __builtin_amdgcn_s_setprio(0);
    softmax_half(s1, p1);
    __builtin_amdgcn_s_setprio(1);
    pv_half(Vs, 1, p1);
    __builtin_amdgcn_s_setprio(0);
  }

  // Row totals over the two lanes of a row: 1/l (0 for an empty row) and the
  // log2-sum-exp (-inf for an empty row).
  __device__ __forceinline__ void finish(float& inv, float& lse2) const {
    const float l_tot = pair_sum(l_run);
    inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    lse2 = l_tot > 0.f ? m_run + __log2f(l_tot) : -INFINITY;
  }
};

// Work-group barrier that waits for nothing by itself.  __syncthreads()
// carries a work-group release fence, and the compiler implements that by
// waiting for every outstanding load, including direct-to-LDS prefetches that
// are meant to stay in flight across the barrier.  Callers wait for what they
// need with s_waitcnt first; the "memory" clobber keeps the compiler from
// moving memory accesses across the barrier.
__device__ __forceinline__ void barrier_keep_loads() { asm volatile("s_barrier" ::: "memory"); }

}  // namespace vico
