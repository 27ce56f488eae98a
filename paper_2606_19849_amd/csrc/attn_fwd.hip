// Bounded chunk-prefill attention for gfx950 (CDNA4).
//
// Computes softmax(Q K^T / sqrt(d)) V for the rows of one visual chunk over
// the keys [sink | W newest history tokens (read through ring slots) |
// chunk keys 0..i] -- the bounded visual attention of ViCoStream (Sec. 3,
// "LLM Prefilling and Decoding"; visibility as in the vision rows of Eq. (4),
// at token granularity, causal inside the chunk).
//
// Mapping onto the hardware
//   * Work-group = 8 waves (two per SIMD, one work-group per CU) = 256 query
//     rows (one key range when split).  Each wave owns 32 rows for the whole
//     key loop; every K/V tile brought into LDS serves all 256 rows.  The
//     rows are 256 tokens of one query head, or packed (token, head) pairs
//     of all query heads of one KV head, token-major (row r: token r / g,
//     head kv*g + r % g) when that takes fewer row tiles: a chunk length
//     that is not a multiple of 256 leaves every query head's last row tile
//     part-empty, and packing leaves one part-filled row tile per KV head
//     instead.  Both forms read the same K/V; the packed one is its own
//     kernel, attn_fwd_packed_kernel.
//   * The tile body (S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_32x32x16_bf16,
//     the exponentiate-first online softmax, two 32-key halves) is WaveTile
//     of attn_common.h, shared with the gathered-query kernel.
//   * K/V tiles: 64 keys, double-buffered in LDS; the next tile's loads
//     are in flight while the current tile is multiplied.  Loads go through
//     buffer resources (one per sink / ring / chunk tensor): a tile that lies
//     inside one segment (and does not cross the ring end) is addressed as a
//     scalar tile base plus a fixed per-thread offset; the few tiles that
//     straddle a boundary resolve each key row (ring slot = ws + k, minus R
//     once past the end) and read all three resources with out-of-range
//     offsets for the wrong ones, which the hardware returns as zero.  Keys
//     past the chunk end read as zero the same way.  No copies are made.
//   * Causal chunk: only tiles that reach past the first row of a wave run the
//     masked variant of the tile body; tiles beyond the last row of a wave are
//     skipped by that wave.  With the bidirectional option (Eq. (4) read
//     literally: a chunk sees all of itself) every row's last key is the
//     chunk's last key, so only the tile holding the chunk end is masked.
//   * Work-groups are renumbered so that consecutive logical ids (the query
//     heads, or the packed row tiles, of one KV head) land on the same XCD
//     and share its L2.
//   * Optional split of the key range (for chunks too small to fill 256 CUs):
//     each split writes fp32 O and log2-sum-exp; a merge kernel combines them.

#include <type_traits>

#include "attn_common.h"

namespace vico {
namespace {

// The kernel body; PACKED selects the packed (token, head) rows.  Inlined
// into one kernel per row form (attn_fwd_kernel, attn_fwd_packed_kernel).
template <int D, bool PACKED>
__device__ __forceinline__ void attn_fwd_body(const AttnArgs& a, int n_rt, int gq) {
  constexpr int BN = kKeyTile;         // keys per tile
  constexpr int BM = kBlockM;          // rows per work-group
  static_assert(kRowBlocks == 1, "one 32-row block per wave (the shared tile body)");
  // LDS tiles: dense rows of 2*D bytes (the direct loads below write each
  // wave's 64 x 16 bytes contiguously), units swizzled as the tile body reads them
  constexpr int UPR = D / 8;           // 16-byte units per row
  constexpr int RBY = D * 2;           // bytes per LDS row
  constexpr int KT = BN * D;           // elements of one K (or V) tile
  constexpr int VT = BN * D;
  constexpr int NW = kThreads / 64;          // waves per work-group
  constexpr int NLD = BN * RBY / 1024 / NW;  // direct 1 KiB loads per wave per tile (K or V)
  constexpr int RPL = 1024 / RBY;            // rows per direct load
  constexpr int NBUF = kBuffers;
  static_assert(NLD * NW * 1024 == BN * RBY, "direct loads cover the tile");
  static_assert(BM == NW * 32, "work-group rows");
  static_assert(NBUF == 2 || NBUF == 3, "two or three LDS buffers");
  static_assert(BN % 64 == 0, "key tiles are whole 64-key sub-tiles");

  // NBUF K/V buffers: tile t lives in buffer t mod NBUF and is loaded NBUF-1
  // tiles ahead.  Separate arrays let the compiler see that reads of one
  // buffer do not wait for the direct loads landing in another.
  __shared__ __attribute__((aligned(16))) uint16_t k_lds0[KT], k_lds1[KT], k_lds2[NBUF > 2 ? KT : 1];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds0[VT], v_lds1[VT], v_lds2[NBUF > 2 ? VT : 1];
  auto kbuf = [&](auto b) __attribute__((always_inline)) -> uint16_t* {
    if constexpr (decltype(b)::value == 0) return k_lds0;
    else if constexpr (decltype(b)::value == 1) return k_lds1;
    else return k_lds2;
  };
  auto vbuf = [&](auto b) __attribute__((always_inline)) -> uint16_t* {
    if constexpr (decltype(b)::value == 0) return v_lds0;
    else if constexpr (decltype(b)::value == 1) return v_lds1;
    else return v_lds2;
  };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int hh = lane >> 5;
  const int C = a.C, S = a.S, SW = a.S + a.Wv;
  const int P = PACKED ? a.pack : 1;   // query heads packed into the rows of a row tile
  const int NR = C * P;                // packed rows of one head group

  // last key visible to chunk token `tok`: its own position (causal), or the
  // chunk's last key when the chunk attends to itself bidirectionally
  auto last_key_of_tok = [&](int tok) __attribute__((always_inline)) {
    return SW + (a.bidir ? C - 1 : min(tok, C - 1));
  };
  // packed row r of a head group is chunk token r / P of query head (group
  // base) + r % P; rows past the group's end stand for its last row
  auto tok_of = [&](int r) __attribute__((always_inline)) { return min(r, NR - 1) / P; };
  // key tiles seen by row tile rt: keys up to its last row's last key
  auto tiles_of = [&](int rt) __attribute__((always_inline)) {
    return (last_key_of_tok(tok_of((rt + 1) * BM - 1)) + BN) / BN;
  };

  // ---- one segment of work: key tiles [t_lo, t_hi) of row tile rt of head
  // group qh of KV head kv (query heads kv*g + qh*P .. + P-1).  `partial`
  // segments write fp32 O and log2-sum-exp to workspace slot `part` (of
  // n_parts) for the merge kernel; others write the output.  All waves of the
  // work-group run the same segments.
  auto segment = [&](int kv, int rt, int qh, int t_lo, int t_hi, int part, int n_parts, bool partial)
      __attribute__((always_inline)) {
  const int h0 = (kv * gq + qh) * P;
  const int row0 = rt * BM;
  const int n_tiles = tiles_of(rt);

  // this wave: packed rows wrow0 + l32; this lane: token tok of head h
  const int wrow0 = row0 + wave * 32;
  const bool wave_active = wrow0 < NR;
  const int wave_first_lim = last_key_of_tok(tok_of(wrow0));      // last key of the wave's first row
  const int wave_last_lim = last_key_of_tok(tok_of(wrow0 + 31));
  const int my_row = min(wrow0 + l32, NR - 1);
  const int tok = my_row / P;
  const int h = h0 + my_row % P;
  const int key_lim = last_key_of_tok(tok);

  // ---- the wave's Q rows and running state.  The Q loads are unconditional:
  // rows past the group's end repeat its last row (the clamped address) and
  // are never stored, and a row's softmax only mixes the two lanes of that row.
  bf16x8 qf[WaveTile<D>::NKS];
  WaveTile<D>::load_q(qf, a.q + ((int64_t)tok * a.Hq + h) * D + hh * 8);

  // ---- tile loader.  Direct load n of wave w fills LDS rows w*BN/4 + n*RPL ..
  // (RPL rows): lane i writes unit i % UPR of row w*BN/4 + n*RPL + i / UPR and
  // fetches the logical unit that belongs there under the swizzle.
  const int rbytes = a.Hkv * D * 2;                            // bytes per token row in HBM
  const rsrc_t rs_sk = make_rsrc(a.sink_k, S * rbytes), rs_sv = make_rsrc(a.sink_v, S * rbytes);
  const rsrc_t rs_rk = make_rsrc(a.ring_k, a.R * rbytes), rs_rv = make_rsrc(a.ring_v, a.R * rbytes);
  const rsrc_t rs_ck = make_rsrc(a.kc, C * rbytes), rs_cv = make_rsrc(a.vc, C * rbytes);
  int ld_row[NLD];                // tile row filled by this lane in load n
  uint32_t ld_ck[NLD], ld_cv[NLD];  // byte offset of the fetched K / V unit inside a token row
#pragma unroll
  for (int n = 0; n < NLD; ++n) {
    const int r = wave * (BN / NW) + n * RPL + lane / UPR;
    const int pu = lane % UPR;
    ld_row[n] = r;
    ld_ck[n] = (uint32_t)(kv * D * 2 + (pu ^ lds_swz_k<D>(r)) * 16);
    ld_cv[n] = (uint32_t)(kv * D * 2 + (pu ^ lds_swz_v<D>(r)) * 16);
  }

  // tile kind (wave-uniform): 0 sink, 1 ring without wrap, 2 chunk, all rows
  // inside the tensor; 3 anything else (segment boundary, ring end, chunk end)
  auto tile_mode = [&](int t, int& row_base) __attribute__((always_inline)) {
    const int k0 = t * BN, k1 = k0 + BN;
    row_base = 0;
    if (k1 <= S) { row_base = k0; return 0; }
    if (k0 >= SW && k1 <= SW + C) { row_base = k0 - SW; return 2; }
    if (k0 >= S && k1 <= SW) {
      int slot0 = a.ws + (k0 - S);
      if (slot0 >= a.R) slot0 -= a.R;
      if (slot0 + BN <= a.R) { row_base = slot0; return 1; }
    }
    return 3;
  };

  // fast tiles: asynchronous direct loads into LDS buffer `buf`
  auto load_tile_direct = [&](auto buf, int mode, int row_base) __attribute__((always_inline)) {
    uint16_t* Ks = kbuf(buf);
    uint16_t* Vs = vbuf(buf);
    const uint16_t* bk = mode == 0 ? a.sink_k : (mode == 1 ? a.ring_k : a.kc);
    const uint16_t* bv = mode == 0 ? a.sink_v : (mode == 1 ? a.ring_v : a.vc);
    const int nb = mode == 0 ? S * rbytes : (mode == 1 ? a.R * rbytes : C * rbytes);
    const rsrc_t rk_ = make_rsrc(bk, nb), rv_ = make_rsrc(bv, nb);
#pragma unroll
    for (int n = 0; n < NLD; ++n) {
      const uint32_t rowoff = (uint32_t)(row_base + ld_row[n]) * (uint32_t)rbytes;
      lds_void* kd = (lds_void*)(Ks + (wave * (BN / NW) + n * RPL) * D);
      lds_void* vd = (lds_void*)(Vs + (wave * (BN / NW) + n * RPL) * D);
      load_lds16(rk_, kd, rowoff + ld_ck[n]);
      load_lds16(rv_, vd, rowoff + ld_cv[n]);
    }
  };

  // other tiles: resolve each key row, read all three tensors (out-of-range
  // offsets return zero), combine, and write the same LDS units.  Synchronous.
  auto load_tile_rows = [&](auto buf, int t) __attribute__((always_inline)) {
    uint16_t* Ks = kbuf(buf);
    uint16_t* Vs = vbuf(buf);
    const int k0 = t * BN;
#pragma unroll
    for (int n = 0; n < NLD; ++n) {
      const int kk = k0 + ld_row[n];
      int slot = a.ws + (kk - S);
      if (slot >= a.R) slot -= a.R;
      const uint32_t o_s = kk < S ? (uint32_t)kk * rbytes : kOutOfRange;
      const uint32_t o_r = (kk >= S && kk < SW) ? (uint32_t)slot * rbytes : kOutOfRange;
      const uint32_t o_c = kk >= SW ? (uint32_t)(kk - SW) * rbytes : kOutOfRange;
      const u32x4 kx = __builtin_amdgcn_raw_buffer_load_b128(rs_sk, o_s + ld_ck[n], 0, 0) |
                       __builtin_amdgcn_raw_buffer_load_b128(rs_rk, o_r + ld_ck[n], 0, 0) |
                       __builtin_amdgcn_raw_buffer_load_b128(rs_ck, o_c + ld_ck[n], 0, 0);
      const u32x4 vx = __builtin_amdgcn_raw_buffer_load_b128(rs_sv, o_s + ld_cv[n], 0, 0) |
                       __builtin_amdgcn_raw_buffer_load_b128(rs_rv, o_r + ld_cv[n], 0, 0) |
                       __builtin_amdgcn_raw_buffer_load_b128(rs_cv, o_c + ld_cv[n], 0, 0);
      const int pos = ld_row[n] * D + (lane % UPR) * 8;
      *(u32x4*)(Ks + pos) = kx;
      *(u32x4*)(Vs + pos) = vx;
    }
  };

  // returns true when the tile went out as asynchronous direct loads
  auto load_tile = [&](auto buf, int t) __attribute__((always_inline)) {
    int row_base;
    const int mode = tile_mode(t, row_base);
    if (mode != 3) {
      load_tile_direct(buf, mode, row_base);
      return true;
    }
    load_tile_rows(buf, t);
    return false;
  };

  uint32_t k_rd[WaveTile<D>::NKS], v_rd[WaveTile<D>::NDB];
  f32x16 o[WaveTile<D>::NDB];
  float m_run, l_run, neg_m;
  WaveTile<D>::start(k_rd, v_rd, o, m_run, l_run, neg_m);
  WaveTile<D> wt{qf, k_rd, v_rd, o, m_run, l_run, neg_m, a.scale_log2};

  // ---- key loop over the buffers: tile t + NBUF - 1 is loaded while tile t is
  // multiplied; one barrier per tile.
  constexpr uint32_t kWaitNewestTile = 0x0F70u | (uint32_t)(2 * NLD);   // vmcnt(2*NLD)
  auto step = [&](auto b, int t) __attribute__((always_inline)) {
    constexpr int B = decltype(b)::value;
    bool async_next = false;
    if (t + NBUF - 1 < t_hi) async_next = load_tile(std::integral_constant<int, (B + NBUF - 1) % NBUF>{}, t + NBUF - 1);
    // the tile body works on 64-key sub-tiles (the operand swizzles only
    // depend on the row modulo 16, so a sub-tile is addressed from its base)
#pragma unroll
    for (int sub = 0; sub < BN / 64; ++sub) {
      const int k0 = t * BN + sub * 64;
      const uint16_t* Ks = kbuf(b) + sub * 64 * D;
      const uint16_t* Vs = vbuf(b) + sub * 64 * D;
      if (wave_active && k0 <= wave_last_lim) {
        if (k0 + 63 > wave_first_lim)
          wt.template tile<true>(Ks, Vs, k0, key_lim, hh);
        else
          wt.template tile<false>(Ks, Vs, k0, key_lim, hh);
      }
    }
    // Tile t + 1 must have landed.  With three buffers the newest tile's
    // direct loads (issued above, if any) may stay in flight.
    if (NBUF == 3 && async_next)
      __builtin_amdgcn_s_waitcnt(kWaitNewestTile);
    else
      __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };
  if (t_lo < t_hi) {
    load_tile(std::integral_constant<int, 0>{}, t_lo);
    if (NBUF == 3 && t_lo + 1 < t_hi) load_tile(std::integral_constant<int, 1>{}, t_lo + 1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int t = t_lo; t < t_hi; t += NBUF) {
      step(std::integral_constant<int, 0>{}, t);
      if (t + 1 < t_hi) step(std::integral_constant<int, 1>{}, t + 1);
      if constexpr (NBUF == 3)
        if (t + 2 < t_hi) step(std::integral_constant<int, 2 % NBUF>{}, t + 2);
    }
  }

  if (!wave_active) return;
  constexpr int NDB = WaveTile<D>::NDB;
  const int row = tok;
  float inv, lse2;
  wt.finish(inv, lse2);
  if (wrow0 + l32 >= NR) return;
  if (!partial) {
    if (a.out_f32) {
      float* op = (float*)a.out + ((int64_t)row * a.Hq + h) * D + hh * 4;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x16& x = o[db];
          *(f32x4*)(op + db * 32 + q4 * 8) =
              f32x4{x[q4 * 4] * inv, x[q4 * 4 + 1] * inv, x[q4 * 4 + 2] * inv, x[q4 * 4 + 3] * inv};
        }
    } else {
      __bf16* op = (__bf16*)a.out + ((int64_t)row * a.Hq + h) * D + hh * 4;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x16& x = o[db];
          *(bf16x4*)(op + db * 32 + q4 * 8) =
              bf16x4{(__bf16)(x[q4 * 4] * inv), (__bf16)(x[q4 * 4 + 1] * inv), (__bf16)(x[q4 * 4 + 2] * inv),
                     (__bf16)(x[q4 * 4 + 3] * inv)};
        }
    }
    if (a.lse && hh == 0) a.lse[(int64_t)h * C + row] = lse2 * kLn2;
  } else {
    float* op = a.ws_o + (((int64_t)part * a.Hq + h) * C + row) * D + hh * 4;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const f32x16& x = o[db];
        *(f32x4*)(op + db * 32 + q4 * 8) =
            f32x4{x[q4 * 4] * inv, x[q4 * 4 + 1] * inv, x[q4 * 4 + 2] * inv, x[q4 * 4 + 3] * inv};
      }
    if (hh == 0) {
      a.ws_lse[((int64_t)part * a.Hq + h) * C + row] = lse2;
      // a row tile that ends in this segment uses no later parts
      if (t_hi == n_tiles)
        for (int p2 = part + 1; p2 < n_parts; ++p2) a.ws_lse[((int64_t)p2 * a.Hq + h) * C + row] = -INFINITY;
    }
  }
  };   // segment

  // ---- schedule
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  if (!a.balanced) {
    // one row tile (one key range of it when split) per work-group
    const int qh = L % gq;
    int rest = L / gq;
    const int rt = n_rt - 1 - rest % n_rt;   // longest row tiles first
    rest /= n_rt;
    const int sp = rest % a.splits;
    const int kv = rest / a.splits;
    const int nt = tiles_of(rt);
    const int t_lo = (int)((int64_t)nt * sp / a.splits);
    const int t_hi = (int)((int64_t)nt * (sp + 1) / a.splits);
    segment(kv, rt, qh, t_lo, t_hi, sp, a.splits, a.splits > 1);
  } else {
    // Balanced: the (row tile, key tile) pairs of all row tiles, in the order
    // kv, row tile (longest first), head group, are cut into gridDim.x equal
    // ranges.  A row tile cut between work-groups is finished by the merge
    // kernel; part = index of the work-group among those covering it.
    const int64_t G = gridDim.x, T = a.total_tiles;
    int64_t pos = (int64_t)L * T / G;
    const int64_t end = (int64_t)(L + 1) * T / G;
    bool first = true;
    while (pos < end) {
      int64_t base = 0;
      int kv = 0, rt = 0, qh = 0, nt = 1;
      for (int k = 0; k < a.Hkv; ++k)
        for (int ri = 0; ri < n_rt; ++ri) {
          const int r = n_rt - 1 - ri;
          const int n = tiles_of(r);
          const int64_t blk = (int64_t)gq * n;
          if (pos >= base && pos < base + blk) {
            kv = k; rt = r; nt = n; qh = (int)((pos - base) / n);
          }
          base += blk;
        }
      // start of the containing row tile in the global order
      int64_t task_start = 0;
      for (int k = 0; k < kv; ++k)
        for (int ri = 0; ri < n_rt; ++ri) task_start += (int64_t)gq * tiles_of(ri);
      for (int ri = 0; ri < n_rt - 1 - rt; ++ri) task_start += (int64_t)gq * tiles_of(n_rt - 1 - ri);
      task_start += (int64_t)qh * nt;
      const int lo = (int)(pos - task_start);
      const int hi = (int)(min(end, task_start + nt) - task_start);
      const int owner = (int)(((task_start + 1) * G - 1) / T);   // work-group holding the row tile's first key tile
      if (!first) __syncthreads();      // the previous segment is done with the LDS buffers
      segment(kv, rt, qh, lo, hi, L - owner, a.splits, true);
      first = false;
      pos = task_start + hi;
    }
  }
}

template <int D>
__global__ __launch_bounds__(kThreads, kWgPerCU) void attn_fwd_kernel(AttnArgs a, int n_rt, int gq) {
  attn_fwd_body<D, false>(a, n_rt, gq);
}

template <int D>
__global__ __launch_bounds__(kThreads, kWgPerCU) void attn_fwd_packed_kernel(AttnArgs a, int n_rt, int gq) {
  attn_fwd_body<D, true>(a, n_rt, gq);
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int grid, hipStream_t stream) {
  const int g = a.Hq / a.Hkv;
  if (a.pack < 1 || g % a.pack != 0) return hipErrorInvalidValue;
  const int gq = g / a.pack;
  const int n_rt = (int)(((int64_t)a.C * a.pack + kBlockM - 1) / kBlockM);
  const dim3 gr(grid), bl(kThreads);
  if (a.pack == 1) {
    if (a.D == 128) hipLaunchKernelGGL(attn_fwd_kernel<128>, gr, bl, 0, stream, a, n_rt, gq);
    else hipLaunchKernelGGL(attn_fwd_kernel<64>, gr, bl, 0, stream, a, n_rt, gq);
  } else {
    if (a.D == 128) hipLaunchKernelGGL(attn_fwd_packed_kernel<128>, gr, bl, 0, stream, a, n_rt, gq);
    else hipLaunchKernelGGL(attn_fwd_packed_kernel<64>, gr, bl, 0, stream, a, n_rt, gq);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (a.splits > 1) return launch_merge(a, stream);   // appends too, when asked
  if (!a.app_rk) return err;
  const AppendArgs ap{a.kc, a.vc, a.app_rk, a.app_rv, a.C, a.R, a.app_p0, a.Hkv * a.D};
  return launch_append(ap, stream);
}

}  // namespace vico
