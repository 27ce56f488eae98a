// Short-query attention over gathered key segments for gfx950 (CDNA4).
//
// Query-side attention of ViCoStream (Sec. 3, query-time decoding; query
// rows of Eq. (4)): the query tokens attend with softmax(Q K~^T / sqrt(d)) V~
// over the keys of the retrieved chunks only.  Here the key set of query row
// i is [sink | store segments, in table order | tail tokens 0 .. T-Lq+i]: the
// segments are slot ranges of a store of past visual K/V (written on the
// device by the top-k kernel, or a ring window split at its end), the tail
// holds the query/answer tokens, of which the query rows are the last Lq.
// With Lq = 1 this is one decode step.
//
// Mapping onto the hardware
//   * A query head group shares its K/V, so the rows of a work-group are
//     packed (token, head) pairs of one KV head: packed row r is query token
//     r / g, head kv*g + r % g.  A decode step (Lq = 1) then still gives g
//     rows per KV head, and a 32-token query 7*32 = 224 rows: one 256-row
//     work-group of 8 waves reads each K/V tile once for all of them.
//   * The tile body (MFMA S^T = K Q^T, online softmax, O^T = V^T P^T with the
//     transposing LDS read, two 32-key halves) is WaveTile of attn_common.h,
//     shared with the chunk prefill kernel.
//   * Keys are walked in 64-key tiles, double-buffered in LDS.  A tile inside
//     the gathered region is loaded straight from HBM into LDS with a slot
//     resolved per lane (the store is one buffer resource, so the rows of a
//     tile may come from several segments); tiles inside the sink or the tail
//     are contiguous; the few tiles that straddle two regions are assembled
//     synchronously.  Segments are clamped to the store, so no access leaves
//     it whatever the table holds.
//   * The segment table (clamped first slots and a prefix sum of lengths) is
//     built in LDS by every work-group; the device-side table never needs a
//     host copy.
//   * Few rows but many keys: the key range is split into parts over the
//     work-groups, merged by the split-merge kernel of the chunk prefill.

#include <type_traits>

#include "attn_common.h"

namespace vico {
namespace {

template <int D>
__global__ __launch_bounds__(kGatherThreads, 1) void attn_gather_kernel(GatherArgs a) {
  constexpr int BN = 64;
  constexpr int BM = kGatherThreads / 64 * 32;
  constexpr int NDB = D / 32;
  constexpr int UPR = D / 8;
  constexpr int RBY = D * 2;
  constexpr int KT = BN * D;
  constexpr int NW = kGatherThreads / 64;
  constexpr int NLD = BN * RBY / 1024 / NW;
  constexpr int RPL = 1024 / RBY;
  constexpr int SEG_PER_THREAD = kMaxSegments / kGatherThreads;
  static_assert(NLD * NW * 1024 == BN * RBY, "direct loads cover the tile");
  static_assert(BM == NW * 32, "one 32-row block per wave");
  static_assert(SEG_PER_THREAD * kGatherThreads == kMaxSegments, "segment table split");

  // NBUF K/V buffers, tile t in buffer t mod NBUF, loaded NBUF-1 tiles ahead:
  // this kernel is bound by HBM, so three tiles stay in flight per work-group.
  // Separate arrays let the compiler see that reads of one buffer do not wait
  // for the direct loads landing in another.
  // (One array per buffer, K then V: the compiler tells apart only a few LDS
  // objects with direct loads in flight, and treats the rest as one.)
  constexpr int NBUF = 4;
  __shared__ __attribute__((aligned(16))) uint16_t kv_lds0[2 * KT], kv_lds1[2 * KT], kv_lds2[2 * KT],
      kv_lds3[2 * KT];
  __shared__ int seg_slot[kMaxSegments];
  __shared__ int seg_pre[kMaxSegments + 1];
  __shared__ int wave_tot[NW];
  auto kbuf = [&](auto b) __attribute__((always_inline)) -> uint16_t* {
    constexpr int B = decltype(b)::value;
    if constexpr (B == 0) return kv_lds0; else if constexpr (B == 1) return kv_lds1;
    else if constexpr (B == 2) return kv_lds2; else return kv_lds3;
  };
  auto vbuf = [&](auto b) __attribute__((always_inline)) -> uint16_t* { return kbuf(b) + KT; };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int hh = lane >> 5;
  const int g = a.Hq / a.Hkv;
  const int NR = g * a.Lq;                 // packed rows per KV head

  // ---- work item
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int rt = L % a.n_rt;
  const int part = (L / a.n_rt) % a.parts;
  const int kv = L / (a.n_rt * a.parts);

  // ---- this lane's packed row
  const int wrow0 = rt * BM + wave * 32;
  const bool wave_active = wrow0 < NR;
  const int my_row = wrow0 + l32;
  const int my_tok = min(my_row, NR - 1) / g;
  const int my_head = kv * g + min(my_row, NR - 1) % g;

  // Q rows as MFMA B fragments.  The loads are unconditional: rows past the
  // end repeat the last row (the clamped address) and are never stored, and
  // a row's softmax only mixes the two lanes of that row.  (Loads under
  // branches, or a later fix-up of their values, leave the compiler unsure
  // whether they completed, and it then waits for every load in flight.)
  // Issued first, so that the wait for the segment table covers them.
  bf16x8 qf[WaveTile<D>::NKS];
  WaveTile<D>::load_q(qf, a.q + ((int64_t)my_tok * a.Hq + my_head) * D + hh * 8);

  // ---- segment table: clamp every segment to the store, prefix-sum lengths
  {
    // every entry of this thread is loaded before any is used (one memory
    // latency); an index past the table reads its last entry and counts as
    // empty.  With no segments the table pointers may be null: no loads.
    int len[SEG_PER_THREAD], run = 0;
    int64_t st[SEG_PER_THREAD];
    int32_t sl[SEG_PER_THREAD];
    if (a.n_segs > 0) {
#pragma unroll
      for (int e = 0; e < SEG_PER_THREAD; ++e) {
        const int ic = min(tid * SEG_PER_THREAD + e, a.n_segs - 1);
        st[e] = a.seg_start[ic];
        sl[e] = a.seg_len[ic];
      }
    }
#pragma unroll
    for (int e = 0; e < SEG_PER_THREAD; ++e) {
      const int i = tid * SEG_PER_THREAD + e;
      int n = 0, slot = 0;
      if (i < a.n_segs) {
        const int64_t lo = st[e] > 0 ? st[e] : 0;
        const int64_t en = st[e] + (int64_t)sl[e];
        const int64_t hi = en < (int64_t)a.cap ? en : (int64_t)a.cap;
        if (hi > lo) { n = (int)(hi - lo); slot = (int)lo; }
      }
      seg_slot[i] = slot;
      len[e] = n;
      run += n;
    }
    // inclusive scan of the per-thread totals: within the wave, then across waves
    int incl = run;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o, 64);
      if (lane >= o) incl += y;
    }
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int base = incl - run;
    for (int w = 0; w < wave; ++w) base += wave_tot[w];
    if (tid == 0) seg_pre[0] = 0;
#pragma unroll
    for (int e = 0; e < SEG_PER_THREAD; ++e) {
      base += len[e];
      seg_pre[tid * SEG_PER_THREAD + e + 1] = base;
    }
    // Q and the table have landed by now; saying so keeps the compiler from
    // waiting for them again, i.e. for every tile load in flight, in the loop.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
    __syncthreads();
  }
  const int S = a.S;
  const int G = __builtin_amdgcn_readfirstlane(seg_pre[a.n_segs]);   // gathered keys (wave-uniform)
  const int SG = S + G;
  const int tail0 = a.T - a.Lq;             // tail tokens before the first query row

  // Gathered key j (0 <= j < G) -> store slot.  Tiles are loaded in key
  // order, so the segment of a tile's first gathered key is found by walking
  // on from the previous tile's (seg_cur, wave-uniform); each lane then walks
  // on from there to its own row's segment (rarely more than one step).
  // Both walks stop below n_segs because seg_pre[n_segs] = G and the index
  // is kept in [seg_pre[seg_cur], G).
  int seg_cur = 0;
  auto seg_advance = [&](int j0) __attribute__((always_inline)) {   // caller: 0 <= j0 < G
    while (seg_pre[seg_cur + 1] <= j0) ++seg_cur;
  };
  auto slot_of = [&](int j) __attribute__((always_inline)) {
    j = min(max(j, seg_pre[seg_cur]), G - 1);
    int s = seg_cur;
    while (seg_pre[s + 1] <= j) ++s;
    return seg_slot[s] + (j - seg_pre[s]);
  };

  // ---- key limits of this wave's rows
  const int key_lim = SG + tail0 + my_tok;                      // last visible key of this lane's row
  const int wave_first_lim = SG + tail0 + min(wrow0, NR - 1) / g;
  const int wave_last_lim = SG + tail0 + min(wrow0 + 31, NR - 1) / g;
  const int rt_last_tok = (min((rt + 1) * BM, NR) - 1) / g;
  const int n_tiles = (SG + tail0 + rt_last_tok + 1 + BN - 1) / BN;
  const int t_lo = (int)((int64_t)n_tiles * part / a.parts);
  const int t_hi = (int)((int64_t)n_tiles * (part + 1) / a.parts);

  // ---- tile loader (see the chunk prefill kernel for the LDS swizzles)
  const int rbytes = a.Hkv * D * 2;
  const rsrc_t rs_sk = make_rsrc(a.sink_k, S * rbytes), rs_sv = make_rsrc(a.sink_v, S * rbytes);
  const rsrc_t rs_gk = make_rsrc(a.store_k, a.cap * rbytes), rs_gv = make_rsrc(a.store_v, a.cap * rbytes);
  const rsrc_t rs_tk = make_rsrc(a.tail_k, a.T * rbytes), rs_tv = make_rsrc(a.tail_v, a.T * rbytes);
  int ld_row[NLD];
  uint32_t ld_ck[NLD], ld_cv[NLD];
#pragma unroll
  for (int n = 0; n < NLD; ++n) {
    const int r = wave * (BN / NW) + n * RPL + lane / UPR;
    const int pu = lane % UPR;
    ld_row[n] = r;
    ld_ck[n] = (uint32_t)(kv * D * 2 + (pu ^ lds_swz_k<D>(r)) * 16);
    ld_cv[n] = (uint32_t)(kv * D * 2 + (pu ^ lds_swz_v<D>(r)) * 16);
  }

  // tile kind (wave-uniform): 0 sink, 1 gathered, 2 tail (all rows inside); 3 mixed
  auto tile_mode = [&](int t) __attribute__((always_inline)) {
    const int k0 = t * BN, k1 = k0 + BN;
    if (k1 <= S) return 0;
    if (k0 >= S && k1 <= SG) return 1;
    if (k0 >= SG && k1 <= SG + a.T) return 2;
    return 3;
  };
  // returns true when the tile went out as asynchronous direct loads
  auto load_tile = [&](auto buf, int t) __attribute__((always_inline)) {
    uint16_t* Ks = kbuf(buf);
    uint16_t* Vs = vbuf(buf);
    const int k0 = t * BN;
    const int mode = tile_mode(t);
    const int j0 = max(k0 - S, 0);
    if (k0 + BN > S && j0 < G) seg_advance(j0);
    if (mode != 3) {
      // select base and size, then build one resource (a select between
      // resources would not stay in scalar registers)
      const uint16_t* bk = mode == 0 ? a.sink_k : (mode == 1 ? a.store_k : a.tail_k);
      const uint16_t* bv = mode == 0 ? a.sink_v : (mode == 1 ? a.store_v : a.tail_v);
      const int nb = (mode == 0 ? S : (mode == 1 ? a.cap : a.T)) * rbytes;
      const rsrc_t rk_ = make_rsrc(bk, nb), rv_ = make_rsrc(bv, nb);
#pragma unroll
      for (int n = 0; n < NLD; ++n) {
        const int kk = k0 + ld_row[n];
        const int row = mode == 0 ? kk : (mode == 1 ? slot_of(kk - S) : kk - SG);
        const uint32_t rowoff = (uint32_t)row * (uint32_t)rbytes;
        lds_void* kd = (lds_void*)(Ks + (wave * (BN / NW) + n * RPL) * D);
        lds_void* vd = (lds_void*)(Vs + (wave * (BN / NW) + n * RPL) * D);
        load_lds16(rk_, kd, rowoff + ld_ck[n]);
        load_lds16(rv_, vd, rowoff + ld_cv[n]);
      }
      return true;
    }
#pragma unroll
    for (int n = 0; n < NLD; ++n) {
      const int kk = k0 + ld_row[n];
      const uint32_t o_s = kk < S ? (uint32_t)kk * rbytes : kOutOfRange;
      const uint32_t o_g = (kk >= S && kk < SG) ? (uint32_t)slot_of(kk - S) * rbytes : kOutOfRange;
      const uint32_t o_t = kk >= SG ? (uint32_t)(kk - SG) * rbytes : kOutOfRange;   // past T: zero
      const u32x4 kx = __builtin_amdgcn_raw_buffer_load_b128(rs_sk, o_s + ld_ck[n], 0, 0) |
                       __builtin_amdgcn_raw_buffer_load_b128(rs_gk, o_g + ld_ck[n], 0, 0) |
                       __builtin_amdgcn_raw_buffer_load_b128(rs_tk, o_t + ld_ck[n], 0, 0);
      const u32x4 vx = __builtin_amdgcn_raw_buffer_load_b128(rs_sv, o_s + ld_cv[n], 0, 0) |
                       __builtin_amdgcn_raw_buffer_load_b128(rs_gv, o_g + ld_cv[n], 0, 0) |
                       __builtin_amdgcn_raw_buffer_load_b128(rs_tv, o_t + ld_cv[n], 0, 0);
      const int pos = ld_row[n] * D + (lane % UPR) * 8;
      *(u32x4*)(Ks + pos) = kx;
      *(u32x4*)(Vs + pos) = vx;
    }
    return false;
  };

  uint32_t k_rd[WaveTile<D>::NKS], v_rd[WaveTile<D>::NDB];
  f32x16 o[WaveTile<D>::NDB];
  float m_run, l_run, neg_m;
  WaveTile<D>::start(k_rd, v_rd, o, m_run, l_run, neg_m);
  WaveTile<D> wt{qf, k_rd, v_rd, o, m_run, l_run, neg_m, a.scale_log2};

  // Key loop.  Step t computes tile t while tiles t+1 .. t+NBUF-1 load; it
  // then waits for tile t+1 only: the direct loads of the newer tiles (each
  // wave issues 2*NLD per asynchronous tile, and loads complete in order)
  // may stay in flight.  `newer_async` = whether tile t+2 went out async.
  // (lgkmcnt(0) too: the synchronous tile path writes LDS with ds_write)
  constexpr uint32_t kWait0 = waitcnt_vm_lgkm0(0);
  constexpr uint32_t kWait1 = waitcnt_vm_lgkm0(2 * NLD);
  constexpr uint32_t kWait2 = waitcnt_vm_lgkm0(4 * NLD);
  static_assert(4 * NLD < 16, "vmcnt immediate");
  auto step = [&](auto b, int t, bool& newer_async) __attribute__((always_inline)) {
    constexpr int B = decltype(b)::value;
    bool an = false;
    if (t + NBUF - 1 < t_hi) an = load_tile(std::integral_constant<int, (B + NBUF - 1) % NBUF>{}, t + NBUF - 1);
    const int k0 = t * BN;
    if (wave_active && k0 <= wave_last_lim) {
      if (k0 + BN - 1 > wave_first_lim)
        wt.template tile<true>(kbuf(b), vbuf(b), k0, key_lim, hh);
      else
        wt.template tile<false>(kbuf(b), vbuf(b), k0, key_lim, hh);
    }
    const int n_newer = (newer_async ? 1 : 0) + (an ? 1 : 0);
    if (n_newer == 2) __builtin_amdgcn_s_waitcnt(kWait2);
    else if (n_newer == 1) __builtin_amdgcn_s_waitcnt(kWait1);
    else __builtin_amdgcn_s_waitcnt(kWait0);
    barrier_keep_loads();
    newer_async = an;
  };
  if (t_lo < t_hi) {
    static_assert(NBUF == 4, "prologue loads three tiles");
    load_tile(std::integral_constant<int, 0>{}, t_lo);
    const bool a1 = t_lo + 1 < t_hi && load_tile(std::integral_constant<int, 1>{}, t_lo + 1);
    const bool a2 = t_lo + 2 < t_hi && load_tile(std::integral_constant<int, 2>{}, t_lo + 2);
    const int n_newer = (a1 ? 1 : 0) + (a2 ? 1 : 0);
    if (n_newer == 2) __builtin_amdgcn_s_waitcnt(kWait2);
    else if (n_newer == 1) __builtin_amdgcn_s_waitcnt(kWait1);
    else __builtin_amdgcn_s_waitcnt(kWait0);
    barrier_keep_loads();
    bool newer_async = a2;
    for (int t = t_lo; t < t_hi; t += NBUF) {
      step(std::integral_constant<int, 0>{}, t, newer_async);
      if (t + 1 < t_hi) step(std::integral_constant<int, 1>{}, t + 1, newer_async);
      if (t + 2 < t_hi) step(std::integral_constant<int, 2>{}, t + 2, newer_async);
      if (t + 3 < t_hi) step(std::integral_constant<int, 3>{}, t + 3, newer_async);
    }
  }

  if (!wave_active || my_row >= NR) return;
  float inv, lse2;
  wt.finish(inv, lse2);
  const int64_t orow = (int64_t)my_tok * a.Hq + my_head;
  if (a.parts == 1) {
    if (a.out_f32) {
      float* op = (float*)a.out + orow * D + hh * 4;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4)
          *(f32x4*)(op + db * 32 + q4 * 8) = f32x4{o[db][q4 * 4] * inv, o[db][q4 * 4 + 1] * inv,
                                                   o[db][q4 * 4 + 2] * inv, o[db][q4 * 4 + 3] * inv};
    } else {
      __bf16* op = (__bf16*)a.out + orow * D + hh * 4;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4)
          *(bf16x4*)(op + db * 32 + q4 * 8) =
              bf16x4{(__bf16)(o[db][q4 * 4] * inv), (__bf16)(o[db][q4 * 4 + 1] * inv),
                     (__bf16)(o[db][q4 * 4 + 2] * inv), (__bf16)(o[db][q4 * 4 + 3] * inv)};
    }
    if (a.lse && hh == 0) a.lse[(int64_t)my_head * a.Lq + my_tok] = lse2 * kLn2;
  } else {
    // partial result of this key range, in the merge kernel's layout (C = Lq)
    const int64_t pr = ((int64_t)part * a.Hq + my_head) * a.Lq + my_tok;
    float* op = a.ws_o + pr * D + hh * 4;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *(f32x4*)(op + db * 32 + q4 * 8) = f32x4{o[db][q4 * 4] * inv, o[db][q4 * 4 + 1] * inv,
                                                 o[db][q4 * 4 + 2] * inv, o[db][q4 * 4 + 3] * inv};
    if (hh == 0) a.ws_lse[pr] = lse2;
  }
}

}  // namespace

hipError_t launch_gather(const GatherArgs& a, hipStream_t stream) {
  const int grid = a.n_rt * a.parts * a.Hkv;
  if (a.D == 128)
    hipLaunchKernelGGL(attn_gather_kernel<128>, dim3(grid), dim3(kGatherThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_gather_kernel<64>, dim3(grid), dim3(kGatherThreads), 0, stream, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || a.parts == 1) return err;
  AttnArgs m{};
  m.out = a.out;
  m.lse = a.lse;
  m.ws_o = a.ws_o;
  m.ws_lse = a.ws_lse;
  m.C = a.Lq;
  m.Hq = a.Hq;
  m.Hkv = a.Hkv;
  m.D = a.D;
  m.splits = a.parts;
  m.out_f32 = a.out_f32;
  return launch_merge(m, stream);
}

}  // namespace vico
