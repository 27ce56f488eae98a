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
 *     frees memory and keeps no state between calls.
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
  VICO_ERR_HIP = -6           /* a HIP runtime call failed */
} vico_status;

enum { VICO_DTYPE_BF16 = 0, VICO_DTYPE_F32 = 1 };

#define VICO_FULL_HISTORY (-1)
#define VICO_SPLIT_BALANCED (-1)

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
 *                  tiles); VICO_SPLIT_BALANCED gives every work-group an equal
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
 * vico_attn_plan -- how vico_chunk_prefill_attn will run for these arguments.
 * Host-only; validates the shape arguments exactly as the attention call does.
 *   *num_splits_out      partial results merged per row (1 = no merge)
 *   *workspace_bytes_out device scratch the call needs (0 when not split)
 * Either output pointer may be NULL.
 */
int vico_attn_plan(int32_t chunk_len, int32_t sink_len, int32_t ring_slots, int64_t hist_len,
                   int64_t window, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                   int32_t num_splits, int32_t* num_splits_out, int64_t* workspace_bytes_out);

/* Workspace size for vico_chunk_prefill_attn; a negative vico_status on bad arguments. */
int64_t vico_attn_workspace_bytes(int32_t chunk_len, int32_t sink_len, int32_t ring_slots, int64_t hist_len,
                                  int64_t window, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t num_splits);

/* Static text for a vico_status value. */
const char* vico_status_str(int status);

/* hipError_t of the last VICO_ERR_HIP returned on the calling thread (0 if none). */
int vico_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* VICO_H */
