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
//     rows of one query head (one key range when split).  Each wave owns 32
//     rows for the whole key loop; every K/V tile brought into LDS serves all
//     256 rows.
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
//     one FMA per logit.  Each half is exponentiated against the running max
//     straight away; the max is only raised (and O rescaled, the half redone)
//     when some lane's sum of probabilities exceeds 2^8, which bounds every
//     probability by 2^8, or while a row has no max yet.  So no row-max
//     reduction sits between the logits and the exponentials.
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
//     heads of one KV head) land on the same XCD and share its L2.
//   * Optional split of the key range (for chunks too small to fill 256 CUs):
//     each split writes fp32 O and log2-sum-exp; a merge kernel combines them.

#include <type_traits>

#include "attn_common.h"

namespace vico {
namespace {

template <int D>
__global__ __launch_bounds__(kThreads, kWgPerCU) void attn_fwd_kernel(AttnArgs a, int n_rt, int g) {
  constexpr int BN = kKeyTile;         // keys per tile
  constexpr int RB = kRowBlocks;       // 32-row blocks per wave
  constexpr int BM = kBlockM;          // rows per work-group
  constexpr int NKS = D / 16;          // k-steps of Q K^T
  constexpr int NDB = D / 32;          // 32-dim blocks of O^T
  // LDS tiles are dense rows of 2*D bytes (the direct loads below write each
  // wave's 64 x 16 bytes contiguously), with 16-byte units permuted inside a
  // row against bank conflicts; the LDS has 64 banks of 4 bytes:
  //   K: unit u of row r sits at u ^ fk(r).  A K fragment read services 16
  //      lanes = 16 consecutive rows at one unit; fk makes them distinct.
  //   V: unit u of row r sits at u ^ fv(r).  A transposing read services 32
  //      lanes = 4 consecutive rows x 4 units; fv spreads the rows apart.
  constexpr int UPR = D / 8;           // 16-byte units per row
  constexpr int RBY = D * 2;           // bytes per LDS row
  constexpr int KT = BN * D;           // elements of one K (or V) tile
  constexpr int VT = BN * D;
  constexpr int NW = kThreads / 64;          // waves per work-group
  constexpr int NLD = BN * RBY / 1024 / NW;  // direct 1 KiB loads per wave per tile (K or V)
  constexpr int RPL = 1024 / RBY;            // rows per direct load
  constexpr int NBUF = kBuffers;
  static_assert(NLD * NW * 1024 == BN * RBY, "direct loads cover the tile");
  static_assert(BM == NW * RB * 32, "work-group rows");
  static_assert(NBUF == 2 || NBUF == 3, "two or three LDS buffers");
  static_assert(BN % 64 == 0, "key tiles are whole 64-key sub-tiles");
  auto fk = [](int r) __attribute__((always_inline)) { return D == 128 ? (r & 15) : ((r >> 1) & 7); };
  auto fv = [](int r) __attribute__((always_inline)) { return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1); };

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
  // last key visible to chunk row `row`: its own position (causal), or the
  // chunk's last key when the chunk attends to itself bidirectionally
  auto last_key_of_row = [&](int row) __attribute__((always_inline)) {
    return SW + (a.bidir ? C - 1 : min(row, C - 1));
  };
  // key tiles seen by row tile rt: keys up to its last row's last key
  auto tiles_of = [&](int rt) __attribute__((always_inline)) {
    return (last_key_of_row((rt + 1) * BM - 1) + BN) / BN;
  };

  // ---- one segment of work: key tiles [t_lo, t_hi) of row tile rt of query
  // head h = kv*g + qh.  `partial` segments write fp32 O and log2-sum-exp to
  // workspace slot `part` (of n_parts) for the merge kernel; others write the
  // output.  All waves of the work-group run the same segments.
  auto segment = [&](int kv, int rt, int qh, int t_lo, int t_hi, int part, int n_parts, bool partial)
      __attribute__((always_inline)) {
  const int h = kv * g + qh;
  const int row0 = rt * BM;
  const int n_tiles = tiles_of(rt);

  // this wave: rows wrow0 + rb*32 + l32, rb < RB
  const int wrow0 = row0 + wave * 32 * RB;
  const bool wave_active = wrow0 < C;
  const int wave_first_lim = last_key_of_row(wrow0);              // last key of the wave's first row
  const int wave_last_lim = last_key_of_row(wrow0 + 32 * RB - 1);
  int key_lim[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) key_lim[rb] = last_key_of_row(wrow0 + rb * 32 + l32);

  // ---- Q rows of this wave as MFMA B fragments (lane: row l32, dims hh*8..+8)
  bf16x8 qf[RB][NKS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = wrow0 + rb * 32 + l32;
    const uint16_t* qp = a.q + ((int64_t)min(row, C - 1) * a.Hq + h) * D + hh * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const u32x4 v = (row < C) ? *(const u32x4*)(qp + ks * 16) : u32x4{0u, 0u, 0u, 0u};
      qf[rb][ks] = __builtin_bit_cast(bf16x8, v);
    }
  }

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
    ld_ck[n] = (uint32_t)(kv * D * 2 + (pu ^ fk(r)) * 16);
    ld_cv[n] = (uint32_t)(kv * D * 2 + (pu ^ fv(r)) * 16);
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

  // per-lane LDS byte offsets of the MFMA operand reads
  //   K fragment (kb, ks): row kb*32 + l32, logical unit 2*ks + hh
  uint32_t k_rd[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) k_rd[ks] = (uint32_t)(l32 * RBY + (((2 * ks) | hh) ^ fk(l32)) * 16);
  //   V^T fragment (db, kp, half): 16-lane group G = lane/16 covers dims
  //   (G%2)*16 .. +15 of a 32-dim block and k-slots (G/2)*8 ..; its lane
  //   4j+q supplies key j of the group's 4 keys (row kp*16 + half*8 +
  //   (G/2)*4 + j), dims 4q .. 4q+3.
  uint32_t v_rd[NDB];
  {
    const int j = (lane & 15) >> 2, q = lane & 3;
    const int r = (lane >> 5) * 4 + j;            // row within the 8-row half-group (fv depends on r mod 4 only)
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int u = db * 4 + ((lane >> 4) & 1) * 2 + (q >> 1);
      v_rd[db] = (uint32_t)(r * RBY + (u ^ fv(r)) * 16 + (q & 1) * 8);
    }
  }

  // ---- running state of this lane's rows (both halves hold the same m)
  f32x16 o[RB][NDB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[rb][db] = f32x16{};
  float m_run[RB], l_run[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) { m_run[rb] = -INFINITY; l_run[rb] = 0.f; }
  const float c = a.scale_log2;

  // Q K^T for one 32-key half of the tile: every K fragment feeds each row block
  auto qk_half = [&](const uint16_t* Ks, int h, f32x16 (&s)[RB]) __attribute__((always_inline)) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) s[rb] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const bf16x8 kf = *(const bf16x8*)((const char*)Ks + h * 32 * RBY + k_rd[ks]);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        s[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[rb][ks], s[rb], 0, 0, 0);
    }
  };
  // causal mask of one half (diagonal tiles only)
  auto mask_half = [&](int k0h, f32x16 (&s)[RB]) __attribute__((always_inline)) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kk = k0h + 8 * (v >> 2) + hh * 4 + (v & 3);
        if (kk > key_lim[rb]) s[rb][v] = -INFINITY;
      }
  };
  // Softmax of one half.  The probabilities are taken against the running
  // max first (exp2, bf16 pack, lane sums), so the exponentials do not wait
  // for a row-max reduction.  While no probability of the wave exceeds 2^8 (a
  // lane's sum bounds each of its 16 terms) that max stays; otherwise, and
  // while a row has no max yet, the max is raised to the half's row max, O and
  // l are rescaled and the half is exponentiated again (rare, wave-uniform).
  auto softmax_half = [&](const f32x16 (&s)[RB], bf16x8 (&pf)[RB][2]) __attribute__((always_inline)) {
    float lsum[RB];
    auto expo = [&](int rb) __attribute__((always_inline)) {
      const float neg_m = (m_run[rb] == -INFINITY) ? 0.f : -m_run[rb];
      float e[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) e[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[rb][v], c, neg_m));
      float s0 = 0.f, s1 = 0.f;      // two chains
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        s0 += e[2 * v];
        s1 += e[2 * v + 1];
      }
#pragma unroll
      for (int kp = 0; kp < 2; ++kp)
#pragma unroll
        for (int j = 0; j < 8; ++j) pf[rb][kp][j] = (__bf16)e[kp * 8 + j];
      lsum[rb] = s0 + s1;
    };
    bool redo = false;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      expo(rb);
      redo |= !(lsum[rb] <= kLaneSumLimit) || m_run[rb] == -INFINITY;
    }
    if (__builtin_amdgcn_ballot_w64(redo)) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[rb][v]);
        // branch-free per lane: a divergent branch here would keep two copies of O
        const float m_new = fmaxf(m_run[rb], pair_max(mx) * c);
        const float alpha = (m_new == m_run[rb]) ? 1.f : __builtin_amdgcn_exp2f(m_run[rb] - m_new);
        l_run[rb] *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db) o[rb][db] *= alpha;
        m_run[rb] = m_new;
        expo(rb);
      }
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) l_run[rb] += lsum[rb];
  };
  // O^T += V^T P^T for one half: every V^T fragment feeds each row block
  auto pv_half = [&](const uint16_t* Vs, int h, const bf16x8 (&pf)[RB][2]) __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        const char* vp = (const char*)Vs + v_rd[db] + (h * 32 + kp * 16) * RBY;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)vp);
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vp + 8 * RBY));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          o[rb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[rb][kp], o[rb][db], 0, 0, 0);
      }
  };

  // One 64-key tile in two 32-key halves, ordered so that the matrix cores
  // multiply one half while the VALU exponentiates the other:
  //   QK(0) | [QK(1) with softmax(0)] [PV(0) with softmax(1)] | PV(1)
  // The wave raises its issue priority while it feeds the matrix cores, so of
  // the two waves sharing a SIMD the one with MFMAs ready goes first and the
  // other's softmax VALU work fills the MFMA shadow.
  auto compute_tile = [&](const uint16_t* Ks, const uint16_t* Vs, int k0, auto mask_tag) __attribute__((always_inline)) {
    constexpr bool MASK = decltype(mask_tag)::value;
    f32x16 s0[RB], s1[RB];
    bf16x8 p0[RB][2], p1[RB][2];
    __builtin_amdgcn_s_setprio(1);
    qk_half(Ks, 0, s0);
    __builtin_amdgcn_s_setprio(0);
    if constexpr (MASK) mask_half(k0, s0);
    __builtin_amdgcn_s_setprio(1);
    qk_half(Ks, 1, s1);
    softmax_half(s0, p0);
    pv_half(Vs, 0, p0);
    if constexpr (MASK) mask_half(k0 + 32, s1);
    __builtin_amdgcn_s_setprio(0);
    softmax_half(s1, p1);
    __builtin_amdgcn_s_setprio(1);
    pv_half(Vs, 1, p1);
    __builtin_amdgcn_s_setprio(0);
  };

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
          compute_tile(Ks, Vs, k0, std::true_type{});
        else
          compute_tile(Ks, Vs, k0, std::false_type{});
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
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = wrow0 + rb * 32 + l32;
    const float l_tot = pair_sum(l_run[rb]);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse2 = l_tot > 0.f ? m_run[rb] + __log2f(l_tot) : -INFINITY;
    if (row >= C) continue;
    if (!partial) {
      if (a.out_f32) {
        float* op = (float*)a.out + ((int64_t)row * a.Hq + h) * D + hh * 4;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            const f32x16& x = o[rb][db];
            *(f32x4*)(op + db * 32 + q4 * 8) =
                f32x4{x[q4 * 4] * inv, x[q4 * 4 + 1] * inv, x[q4 * 4 + 2] * inv, x[q4 * 4 + 3] * inv};
          }
      } else {
        __bf16* op = (__bf16*)a.out + ((int64_t)row * a.Hq + h) * D + hh * 4;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            const f32x16& x = o[rb][db];
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
          const f32x16& x = o[rb][db];
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
  }
  };   // segment

  // ---- schedule
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  if (!a.balanced) {
    // one row tile (one key range of it when split) per work-group
    const int qh = L % g;
    int rest = L / g;
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
    // kv, row tile (longest first), query head, are cut into gridDim.x equal
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
          const int64_t blk = (int64_t)g * n;
          if (pos >= base && pos < base + blk) {
            kv = k; rt = r; nt = n; qh = (int)((pos - base) / n);
          }
          base += blk;
        }
      // start of the containing row tile in the global order
      int64_t task_start = 0;
      for (int k = 0; k < kv; ++k)
        for (int ri = 0; ri < n_rt; ++ri) task_start += (int64_t)g * tiles_of(ri);
      for (int ri = 0; ri < n_rt - 1 - rt; ++ri) task_start += (int64_t)g * tiles_of(n_rt - 1 - ri);
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

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int grid, hipStream_t stream) {
  const int g = a.Hq / a.Hkv;
  const int n_rt = (a.C + kBlockM - 1) / kBlockM;
  if (a.D == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3(grid), dim3(kThreads), 0, stream, a, n_rt, g);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3(grid), dim3(kThreads), 0, stream, a, n_rt, g);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || a.splits == 1) return err;
  return launch_merge(a, stream);
}

}  // namespace vico
