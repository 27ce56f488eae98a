/*
 * vico.h -- C ABI of the bounded chunk-prefill attention library for AMD
 * Instinct MI355X (gfx950).
 *
 * The operation (ViCoStream, Sec. 3, "LLM Prefilling and Decoding"): a
 * streaming VideoLLM prefills each incoming chunk of retained visual tokens
 * with attention bounded to recent visual history,
 *     Attn = softmax(Q K_hat^T / sqrt(d)) V_hat,
 * instead of the whole accumulated stream; the vision rows of the additive
 * mask of Eq. (4) fix which keys are visible.  This library realises the
 * visible set at token granularity as
 *     [ sink prefix (S tokens) | W newest history tokens | chunk tokens 0..i ]
 * for chunk row i (causal inside the chunk), under grouped-query attention,
 * with the history held in a ring-buffer KV cache of R token slots.  A
 * full-history mode (window = VICO_FULL_HISTORY) is the unbounded streaming
 * prefill the paper compares against.
 *
 * Conventions shared by every entry point
 *   - Tensors are dense, row-major, bfloat16 unless stated otherwise, in
 *     device memory owned by the caller.  The library never allocates or
 *     frees memory and keeps no state between calls, except the fixed
 *     device array of vico_gather_attn_noalloc (below).
 *   - Token-major layouts:  Q and O are [tokens][num_q_heads][head_dim];
 *     K/V (chunk, sink, ring) are [tokens][num_kv_heads][head_dim].
 *   - Ring slot p % ring_slots holds linear history token p.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream)
 *     and the call returns without waiting for it.  Calls on one stream run
 *     in issue order; ordering across streams is the caller's business.
 *   - Every device pointer must be 16-byte aligned (lse_out: 4-byte).
 *   - Host-detectable errors return a negative vico_status before anything
 *     is enqueued; nothing is written.  VICO_ERR_HIP reports a failed HIP
 *     call (launch error); vico_last_hip_error() gives its hipError_t.
 *   - head_dim must be 64 or 128.
 */
#ifndef VICO_H
#define VICO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  VICO_OK = 0,
  VICO_ERR_INVALID_ARG = -1,  /* bad count, NULL pointer, overlapping buffers */
  VICO_ERR_UNSUPPORTED = -2,  /* head_dim or dtype the kernels do not cover */
  VICO_ERR_CAPACITY = -3,     /* ring too small for the window or the chunk */
  VICO_ERR_MISALIGNED = -4,   /* pointer not 16-byte (lse_out: 4-byte) aligned */
  VICO_ERR_WORKSPACE = -5,    /* workspace missing or smaller than required */
  VICO_ERR_HIP = -6,          /* a HIP runtime call failed */
  VICO_ERR_SCRATCH = -7       /* needs more than the fixed VICO_NOALLOC_SCRATCH_BYTES */
} vico_status;

enum { VICO_DTYPE_BF16 = 0, VICO_DTYPE_F32 = 1 };

#define VICO_FULL_HISTORY (-1)
#define VICO_SPLIT_BALANCED (-1)
/* flags of the _ex entry points */
#define VICO_ATTN_BIDIRECTIONAL 1  /* every chunk row sees the whole chunk (no causal mask) */
#define VICO_ATTN_APPEND 2         /* then append the chunk's K/V to the ring (as vico_kv_append) */

/*
 * vico_kv_append -- append a chunk's K/V to the ring-buffer visual cache.
 *
 * The paper bounds the cache a chunk can see (Sec. 3, "LLM Prefilling and
 * Decoding"); a ring of ring_slots token slots keeps exactly the newest
 * tokens.  For j in [0, chunk_len):
 *     ring_k[(hist_len + j) % ring_slots] = k_chunk[j]
 *     ring_v[(hist_len + j) % ring_slots] = v_chunk[j]
 * as a bit copy of rows of num_kv_heads * head_dim bf16 values.
 *
 *   k_chunk, v_chunk  [chunk_len][num_kv_heads][head_dim] bf16, device, read
 *   ring_k, ring_v    [ring_slots][num_kv_heads][head_dim] bf16, device, written
 *   hist_len          linear count of tokens appended before this chunk (>= 0)
 *
 * chunk_len == 0 is a no-op.  chunk_len > ring_slots -> VICO_ERR_CAPACITY.
 * Chunk and ring buffers must not overlap (VICO_ERR_INVALID_ARG).
 * To let a chunk attend to the window that its own append would overwrite,
 * enqueue vico_chunk_prefill_attn for the chunk before its append.
 */
int vico_kv_append(const void* k_chunk, const void* v_chunk, int32_t chunk_len,
                   void* ring_k, void* ring_v, int32_t ring_slots, int64_t hist_len,
                   int32_t num_kv_heads, int32_t head_dim, void* stream);

/*
 * vico_chunk_prefill_attn -- bounded chunk-prefill attention.
 *
 * Sec. 3 ("LLM Prefilling and Decoding") and Eq. (4), at token granularity:
 * with Wv = min(window, hist_len) (hist_len if window == VICO_FULL_HISTORY)
 * and g = num_q_heads / num_kv_heads, output row i of query head h is
 *     out[i][h] = sum_j softmax_j(scale * <q[i][h], k_j>) v_j
 * over the keys j of KV head h / g in
 *     sink[0 .. sink_len)  ++  history[hist_len - Wv .. hist_len)  ++  chunk[0 .. i]
 * where history token p is read from ring slot p % ring_slots.
 *
 *   q              [chunk_len][num_q_heads][head_dim] bf16, device (post-RoPE)
 *   k_chunk,v_chunk[chunk_len][num_kv_heads][head_dim] bf16, device
 *   sink_k,sink_v  [sink_len][num_kv_heads][head_dim] bf16; NULL iff sink_len == 0
 *   ring_k,ring_v  [ring_slots][num_kv_heads][head_dim] bf16; may be NULL iff Wv == 0
 *   window         visible history tokens (>= 0) or VICO_FULL_HISTORY
 *   softmax_scale  <= 0 selects 1/sqrt(head_dim)
 *   out            [chunk_len][num_q_heads][head_dim], out_dtype BF16 (rounded to
 *                  nearest even) or F32
 *   lse_out        NULL or [num_q_heads][chunk_len] fp32: natural-log sum of
 *                  exp(scale * q.k) over the visible keys of each row
 *   num_splits     0: the library picks the schedule; n > 0 splits every row
 *                  tile's key range into n parts (clamped to the number of key
 *                  tiles and to 16); VICO_SPLIT_BALANCED gives every work-group an equal
 *                  share of all key tiles of all row tiles.  Split or shared
 *                  row tiles are combined by a log-sum-exp merge.  Results
 *                  agree up to rounding for every choice.
 *   workspace      device scratch of at least vico_attn_workspace_bytes(...) bytes
 *                  for the same arguments; may be NULL when that size is 0.
 *
 * Arithmetic: bf16 MFMA products with fp32 accumulation, fp32 online softmax,
 * probabilities rounded to bf16 for the P.V product.
 * Errors: Wv > ring_slots -> VICO_ERR_CAPACITY (history already evicted);
 * chunk_len == 0 is a no-op.  The window is read through the ring before
 * this chunk's own append; the caller orders the two calls on the stream.
 */
int vico_chunk_prefill_attn(const void* q, const void* k_chunk, const void* v_chunk, int32_t chunk_len,
                            const void* sink_k, const void* sink_v, int32_t sink_len,
                            const void* ring_k, const void* ring_v, int32_t ring_slots, int64_t hist_len,
                            int64_t window, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                            float softmax_scale, void* out, int32_t out_dtype, float* lse_out,
                            int32_t num_splits, void* workspace, int64_t workspace_bytes, void* stream);

/*
 * vico_chunk_prefill_attn_ex -- vico_chunk_prefill_attn with options.
 *
 * flags = 0 is vico_chunk_prefill_attn.  VICO_ATTN_BIDIRECTIONAL: the
 * additive mask of Eq. (4) read literally -- a vision token sees every token
 * of the chunks in its window, its own chunk included -- so row i sees
 * chunk[0 .. chunk_len) instead of chunk[0 .. i].  VICO_ATTN_APPEND: after
 * attending, the call also does what vico_kv_append(k_chunk, v_chunk, ...,
 * hist_len) would (the ring of Sec. 3 advances by the chunk), after every
 * read of the window: the split-merge kernel copies the chunk alongside the
 * merge, so a split call saves a launch; without a split the copy is its own
 * launch.  It needs ring_k/ring_v, chunk_len <= ring_slots, and chunk buffers
 * that do not overlap the ring (as vico_kv_append).  Other bits are invalid.
 * Use vico_attn_plan_ex with the same flags for the workspace size.
 *
 * The paper's window is whole chunks (the most recent acn chunks, the
 * staircase band of Eq. (4)); pass window = vico_acn_window(...) to get it
 * exactly from the caller's table of chunk start positions.
 */
int vico_chunk_prefill_attn_ex(const void* q, const void* k_chunk, const void* v_chunk, int32_t chunk_len,
                               const void* sink_k, const void* sink_v, int32_t sink_len,
                               const void* ring_k, const void* ring_v, int32_t ring_slots, int64_t hist_len,
                               int64_t window, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                               float softmax_scale, void* out, int32_t out_dtype, float* lse_out,
                               int32_t num_splits, int32_t flags, void* workspace, int64_t workspace_bytes,
                               void* stream);

/*
 * vico_acn_window -- visible history of chunk t under the chunk-granular
 * window of Sec. 3 / Eq. (4): the vision rows of chunk t see chunks
 * t-acn .. t, i.e. the history chunks max(0, t-acn) .. t-1, which is
 *     chunk_starts[t] - chunk_starts[max(0, t - acn)]
 * tokens (acn < 0: chunk_starts[t], the whole history).
 *   chunk_starts  HOST array of num_chunks linear start positions (the number
 *                 of tokens appended before each chunk), non-decreasing
 * Returns the window in tokens, or a negative vico_status (t outside the
 * table, NULL table, decreasing starts).  Host-only arithmetic.
 */
int64_t vico_acn_window(const int64_t* chunk_starts, int32_t num_chunks, int32_t t, int32_t acn);

/*
 * vico_attn_plan -- how vico_chunk_prefill_attn will run for these arguments.
 * Host-only; validates the shape arguments exactly as the attention call does.
 *   *num_splits_out      partial results merged per row (1 = no merge)
 *   *workspace_bytes_out device scratch the call needs (0 when not split)
 * Either output pointer may be NULL.
 */
int vico_attn_plan(int32_t chunk_len, int32_t sink_len, int32_t ring_slots, int64_t hist_len,
                   int64_t window, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                   int32_t num_splits, int32_t* num_splits_out, int64_t* workspace_bytes_out);

/* vico_attn_plan for vico_chunk_prefill_attn_ex with the given flags. */
int vico_attn_plan_ex(int32_t chunk_len, int32_t sink_len, int32_t ring_slots, int64_t hist_len,
                      int64_t window, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                      int32_t num_splits, int32_t flags, int32_t* num_splits_out, int64_t* workspace_bytes_out);

/* Workspace size for vico_chunk_prefill_attn; a negative vico_status on bad arguments. */
int64_t vico_attn_workspace_bytes(int32_t chunk_len, int32_t sink_len, int32_t ring_slots, int64_t hist_len,
                                  int64_t window, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t num_splits);

/* ------------------------------------------------------------------------
 * Query-side retrieval (Sec. 3, query-time decoding; query rows of Eq. (4)).
 * The query tokens and each visual chunk's retained tokens are averaged
 * into one representative feature each; chunks are ranked by the cosine of
 * the two; only the retrieved chunks' keys and values are visible to the
 * query tokens.  A typical query: vico_token_mean on the query embeddings,
 * vico_chunk_scores over the feature table, vico_topk_chunks (which also
 * writes the store segments), then vico_gather_attn per layer -- no host
 * synchronisation anywhere in between.
 * ------------------------------------------------------------------------ */

/*
 * vico_token_mean -- representative feature: out[c] = (1/L) sum_t x[t][c].
 *
 *   x        [num_tokens][feat_dim] bf16, device (LLM input embeddings of a
 *            chunk's retained tokens, or of the query tokens)
 *   out      [feat_dim] fp32, device, written
 * num_tokens >= 1; feat_dim a positive multiple of 8.  fp32 accumulation in a
 * fixed order (results repeat bit for bit).  x 16-byte, out 16-byte aligned.
 */
int vico_token_mean(const void* x, int32_t num_tokens, int32_t feat_dim, float* out, void* stream);

/*
 * vico_chunk_scores -- s_i = <q, c_i> / (|q| |c_i|) (the retrieval equation
 * of Sec. 3), fp32.  A zero vector on either side scores 0.
 *
 *   query_feat  [feat_dim] fp32, device
 *   chunk_feat  [num_chunks][feat_dim] fp32, device (one row per stored chunk)
 *   scores      [num_chunks] fp32, device, written
 * feat_dim a positive multiple of 8; num_chunks >= 0 (0 is a no-op).
 */
int vico_chunk_scores(const float* query_feat, const float* chunk_feat, int32_t num_chunks, int32_t feat_dim,
                      float* scores, void* stream);

/*
 * vico_topk_chunks -- the retrieved set: the top_k chunks by score among
 * those with score >= min_score (pass -INFINITY for plain top-k; a finite
 * value is the threshold tau_q of the training mask of Eq. (4)).  Equal
 * scores rank the earlier chunk first; NaN scores are never selected.
 * The selected chunks are written in ascending chunk order (stream order):
 *
 *   out_chunks  [top_k] int32, device: chunk indices, then -1 padding
 *   out_scores  [top_k] fp32, device: their scores, then -inf padding
 *   out_count   [1] int32, device: number selected = min(top_k, candidates)
 *   chunk_start [num_chunks] int64, chunk_len [num_chunks] int32, device:
 *               the store slot range of every chunk; when both are non-NULL
 *               the call also writes the segment table of the selection,
 *   seg_start   [top_k] int64, seg_len [top_k] int32, device (zero padding),
 *               ready to be passed to vico_gather_attn.
 * 1 <= top_k <= 2048, num_chunks >= 0.  One work-group; cost grows with
 * num_chunks (five passes over the scores).
 */
int vico_topk_chunks(const float* scores, int32_t num_chunks, int32_t top_k, float min_score,
                     const int64_t* chunk_start, const int32_t* chunk_len, int32_t* out_chunks,
                     float* out_scores, int64_t* seg_start, int32_t* seg_len, int32_t* out_count, void* stream);

/*
 * vico_gather_attn -- attention of short query rows over gathered chunks.
 *
 * Attn_q = softmax(Q_q K~^T / sqrt(d)) V~ (Sec. 3) where K~, V~ are built
 * from the retrieved chunks.  With g = num_q_heads / num_kv_heads, the query
 * rows are the last q_len of tail_len tail tokens (the query, or the
 * answer tokens generated so far), and row i of query head h attends to the
 * keys of KV head h / g in
 *     sink[0 .. sink_len) ++ store[segment 0] ++ ... ++ store[segment n-1]
 *                         ++ tail[0 .. tail_len - q_len + i]
 * where segment s is store slots [seg_start[s], seg_start[s] + seg_len[s]).
 * q_len = 1 is one decode step; a ring window is passed as one or two
 * segments of the ring.
 *
 *   q              [q_len][num_q_heads][head_dim] bf16, device
 *   tail_k,tail_v  [tail_len][num_kv_heads][head_dim] bf16, device
 *   sink_k,sink_v  [sink_len][num_kv_heads][head_dim]; NULL iff sink_len == 0
 *   store_k,store_v[store_slots][num_kv_heads][head_dim] bf16, device
 *   seg_start      [num_segments] int64, device (8-byte aligned)
 *   seg_len        [num_segments] int32, device (4-byte aligned)
 *   keys_hint      expected total segment length; only sets how the key range
 *                  is split over work-groups (any value gives the same result)
 *   out, out_dtype, lse_out, softmax_scale: as for vico_chunk_prefill_attn
 *                  ([q_len][num_q_heads][head_dim], [num_q_heads][q_len])
 *   num_splits     0: library's choice; n > 0: key range in n parts (<= 64)
 *   workspace      at least the bytes vico_gather_plan reports
 *
 * The table lives in device memory (vico_topk_chunks writes it), so it is
 * checked on the device: every segment is clipped to [0, store_slots), and
 * the parts outside the store are not attended to.  0 <= num_segments <=
 * 2048; num_segments * store_slots + sink_len + tail_len <= 2^30;
 * 1 <= q_len <= tail_len.  Arithmetic as for vico_chunk_prefill_attn.
 */
int vico_gather_attn(const void* q, int32_t q_len, const void* tail_k, const void* tail_v, int32_t tail_len,
                     const void* sink_k, const void* sink_v, int32_t sink_len, const void* store_k,
                     const void* store_v, int32_t store_slots, const int64_t* seg_start, const int32_t* seg_len,
                     int32_t num_segments, int64_t keys_hint, int32_t num_q_heads, int32_t num_kv_heads,
                     int32_t head_dim, float softmax_scale, void* out, int32_t out_dtype, float* lse_out,
                     int32_t num_splits, void* workspace, int64_t workspace_bytes, void* stream);

/*
 * vico_gather_plan -- key-range parts and workspace of vico_gather_attn for
 * these arguments (host-only; validates them as the call does).
 */
int vico_gather_plan(int32_t q_len, int32_t tail_len, int32_t sink_len, int32_t store_slots,
                     int32_t num_segments, int64_t keys_hint, int32_t num_q_heads, int32_t num_kv_heads,
                     int32_t head_dim, int32_t num_splits, int32_t* num_splits_out, int64_t* workspace_bytes_out);

/*
 * vico_gather_attn_noalloc -- vico_gather_attn for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, result and kernels as
 * vico_gather_attn, without the workspace: the key-range partials go to a
 * fixed device array of VICO_NOALLOC_SCRATCH_BYTES (64 MiB) inside the
 * library.  The caller still owns q, K/V, the segment table, out and lse_out.
 *
 *   - A call whose plan (vico_gather_plan) needs more than
 *     VICO_NOALLOC_SCRATCH_BYTES returns VICO_ERR_SCRATCH and enqueues
 *     nothing.  The library's own split (num_splits = 0) needs at most
 *     33.9 MB at head_dim 128 for any query length and head count, so only
 *     an explicit num_splits can exceed it (a 7B decode step needs 0.9 MB).
 *   - Each GPU gets its own copy of the array, created with the library's
 *     code object on that GPU and held until the process ends.  Its address
 *     is looked up on the first call made with that device current (before
 *     capturing a graph, make one eager call on the device).
 *   - Calls no hipMalloc, hipFree, hipMemset or copy; it only launches kernels.
 *   - All calls on one GPU share its array: two calls that may run at the
 *     same time on that GPU (different streams, no ordering between them)
 *     race and give wrong results.  Calls ordered on one stream are fine;
 *     every partial is written before it is read, so nothing is cleared.
 */
#define VICO_NOALLOC_SCRATCH_BYTES (64ll << 20)
int vico_gather_attn_noalloc(const void* q, int32_t q_len, const void* tail_k, const void* tail_v, int32_t tail_len,
                             const void* sink_k, const void* sink_v, int32_t sink_len, const void* store_k,
                             const void* store_v, int32_t store_slots, const int64_t* seg_start,
                             const int32_t* seg_len, int32_t num_segments, int64_t keys_hint, int32_t num_q_heads,
                             int32_t num_kv_heads, int32_t head_dim, float softmax_scale, void* out,
                             int32_t out_dtype, float* lse_out, int32_t num_splits, void* stream);

/*
 * vico_temporal_drop -- chunk-level temporal token dropping (Sec. 3, "Token
 * Dropping", the pairwise-similarity and drop equations).
 *
 * For each of num_chunks consecutive chunks of C = frames_per_chunk frames
 * and each spatial position p, the cosine of the frames' tokens at p is taken
 * for every frame pair i < j; p is dropped when all of them exceed tau
 * (strictly), and the chunk's first frame is always kept (the anchor), so a
 * dropped position keeps only its frame-1 token.  With C = 1 every frame is
 * compared with the frame before it (prev_frame for the first one; with
 * prev_frame NULL the first frame is kept whole) and there is no anchor.
 * Cosines are fp32 sums of the bf16 products; a zero vector scores 0.
 *
 *   frames      [num_chunks][C][tokens_per_frame][feat_dim] bf16, device
 *   prev_frame  [tokens_per_frame][feat_dim] bf16 or NULL (C = 1 only; ignored otherwise)
 *   keep        [num_chunks][tokens_per_frame] uint8, written: 1 = position kept
 *   sim         NULL or [num_chunks][tokens_per_frame] fp32, written: the
 *               smallest pairwise cosine (C = 1: the cosine with the previous
 *               frame, -2 where there is none); keep == !(sim > tau) exactly
 *   out_tokens  NULL or capacity for num_chunks*C*tokens_per_frame rows of
 *               feat_dim bf16: the retained tokens, in stream order (chunk,
 *               frame, position), bit copies of the inputs
 *   out_index   [num_chunks*C*tokens_per_frame] int32: flat source row
 *               (chunk*C + frame)*tokens_per_frame + position of each
 *               retained token, in the same order
 *   out_count   [1] int32: number of retained tokens
 *   workspace   NULL, or device scratch of at least
 *               vico_temporal_drop_workspace_bytes(...) bytes, 8-byte aligned,
 *               overlapping no other argument (VICO_ERR_WORKSPACE if smaller,
 *               VICO_ERR_MISALIGNED if not aligned); its contents need no
 *               initialisation and are meaningless afterwards.  Calls that share
 *               one workspace must be ordered (same stream, or synchronised).
 * 1 <= C <= 8, feat_dim a positive multiple of 8, fewer than 2^31 rows;
 * num_chunks == 0 is a no-op.
 *
 * Schedules (same results, bit for bit):
 *   workspace NULL, or a shape the single pass does not cover (workspace
 *   bytes 0): two passes -- similarities and flags, then ranking and copying,
 *   which reads the retained rows a second time.
 *   otherwise: one pass in which each token row is read once and stored at
 *   its final place; its work-groups share their counts of kept positions
 *   through the workspace (words tagged per call, so no zeroing is needed).
 *   A work-group that waits more than 200 us for another one's count
 *   (environment variable VICO_DROP_WAIT_US, read at every call) recomputes it from
 *   the frames instead, so the results never depend on scheduling.  Under
 *   HIP graph capture the call takes the two passes (the single pass tags its
 *   words per call, and a replayed graph would repeat the tag).
 */
int vico_temporal_drop(const void* frames, int32_t num_chunks, int32_t frames_per_chunk, int32_t tokens_per_frame,
                       int32_t feat_dim, float tau, const void* prev_frame, uint8_t* keep, float* sim,
                       void* out_tokens, int32_t* out_index, int32_t* out_count, void* workspace,
                       int64_t workspace_bytes, void* stream);

/*
 * vico_temporal_drop_workspace_bytes -- workspace bytes of the single-pass
 * schedule of vico_temporal_drop for these sizes: 0 where that schedule does
 * not apply (num_chunks == 0 or above 256, tokens_per_frame > 1024, or
 * feat_dim above 512 * min(8, 32 / max(C, 2)) with integer division: 4096 up
 * to C = 4, then 3072, 2560, 2048, 2048), VICO_ERR_INVALID_ARG for sizes
 * vico_temporal_drop rejects.  128 bytes per chunk and 8 per tile of 4
 * positions: num_chunks * (128 + 8 * ceil(tokens_per_frame / 4)).
 */
int64_t vico_temporal_drop_workspace_bytes(int32_t num_chunks, int32_t frames_per_chunk, int32_t tokens_per_frame,
                                           int32_t feat_dim);

/* Static text for a vico_status value. */
const char* vico_status_str(int status);

/* hipError_t of the last VICO_ERR_HIP returned on the calling thread (0 if none). */
int vico_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* VICO_H */
