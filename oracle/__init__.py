"""fp64 CPU oracle for bounded chunk-prefill attention and the ring KV cache.

TEST INFRASTRUCTURE ONLY.  Nothing in the product library imports, calls or
links this package; only the tests, the smoke check and the CPU-baseline leg
of the benchmark do.  It shares no code with the HIP path.

What it computes (paper, Sec. 3, "LLM Prefilling and Decoding"): each
incoming visual chunk attends with softmax(Q K^T / sqrt(d)) V over a bounded
set of keys -- here a fixed sink prefix, the W most recent history tokens and
the chunk itself under a causal mask -- instead of the whole accumulated
history.  The visibility rules restate the vision rows of the additive mask of
Eq. (4) at token granularity.  Readings where the paper is silent are listed
in the module docstrings.

Modules
  bf16       -- widen bfloat16 bit patterns to float64 exactly
  attention  -- exact masked softmax attention (blocked and per-row forms)
  ring       -- linear-history model of the ring-buffer KV cache
  merge      -- log-sum-exp merge of attention over disjoint key sets
  retrieval  -- query-side chunk retrieval (token means, cosine scores,
                top-k selection) and attention over the retrieved chunks
  token_drop -- chunk-level temporal token dropping (pairwise cosine over
                frames, anchor frame) and the retained-token order

Parity status: every function here is pinned by tests in
tests/test_oracle_pins.py, tests/test_oracle_retrieval_pins.py,
tests/test_oracle_acn_pins.py and tests/test_oracle_drop_pins.py against library routines, closed forms,
invariants and brute force; none is "parity unpinned".
"""
from .bf16 import bf16_bits_to_f64
from .attention import (
    softmax_attention,
    chunk_prefill_attention,
    chunk_prefill_attention_rowloop,
    visible_window,
    kv_head_of,
    acn_window,
)
from .ring import RingModel
from .merge import lse_merge
from .retrieval import token_mean, cosine_scores, select_chunks, chunk_segments, gather_attention
from .token_drop import temporal_drop, retained_index, gather_tokens, NO_COMPARISON

__all__ = [
    "bf16_bits_to_f64",
    "softmax_attention",
    "chunk_prefill_attention",
    "chunk_prefill_attention_rowloop",
    "visible_window",
    "kv_head_of",
    "acn_window",
    "RingModel",
    "lse_merge",
    "token_mean",
    "cosine_scores",
    "select_chunks",
    "chunk_segments",
    "gather_attention",
    "temporal_drop",
    "retained_index",
    "gather_tokens",
    "NO_COMPARISON",
]
