"""Bounded chunk-prefill attention and ring-buffer KV append for MI355X (gfx950).

The hot path of ViCoStream's bounded visual attention (Sec. 3, "LLM
Prefilling and Decoding"): each video chunk's retained visual tokens attend
to a sink prefix, the W newest cached visual tokens and themselves
(causally) under grouped-query attention; the chunk's K/V then enter a
ring-buffer cache.  Query-side retrieval (token means, cosine scores, top-k
chunks) and attention of short queries or decode steps over the retrieved
chunks complete the query path; temporal token dropping thins each chunk's
tokens before they reach the LLM.  All arithmetic runs in the hand-written HIP
kernels of libvico.so (C ABI in include/vico.h); this package only marshals
arguments.
"""
from ._binding import (
    VICO_DTYPE_BF16,
    VICO_DTYPE_F32,
    VICO_FULL_HISTORY,
    VICO_SPLIT_BALANCED,
    VICO_ATTN_BIDIRECTIONAL,
    VICO_ATTN_APPEND,
    VICO_NOALLOC_SCRATCH_BYTES,
    VicoError,
    load_library,
    header_functions,
    vico_attn_plan,
    vico_attn_workspace_bytes,
    vico_chunk_prefill_attn,
    vico_kv_append,
    vico_token_mean,
    vico_chunk_scores,
    vico_topk_chunks,
    vico_gather_plan,
    vico_gather_attn,
    vico_gather_attn_noalloc,
    vico_acn_window,
    vico_temporal_drop,
    vico_temporal_drop_workspace_bytes,
)

__all__ = [
    "VICO_DTYPE_BF16",
    "VICO_DTYPE_F32",
    "VICO_FULL_HISTORY",
    "VICO_SPLIT_BALANCED",
    "VICO_ATTN_BIDIRECTIONAL",
    "VICO_ATTN_APPEND",
    "VICO_NOALLOC_SCRATCH_BYTES",
    "VicoError",
    "load_library",
    "header_functions",
    "vico_attn_plan",
    "vico_attn_workspace_bytes",
    "vico_chunk_prefill_attn",
    "vico_kv_append",
    "vico_token_mean",
    "vico_chunk_scores",
    "vico_topk_chunks",
    "vico_gather_plan",
    "vico_gather_attn",
    "vico_gather_attn_noalloc",
    "vico_acn_window",
    "vico_temporal_drop",
    "vico_temporal_drop_workspace_bytes",
]
