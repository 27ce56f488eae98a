"""Query-side chunk retrieval and attention over the retrieved chunks, float64.

Definitions followed (paper, Sec. 3, "LLM Prefilling and Decoding", query-time
decoding, and the query rows of the additive mask of Eq. (4)):

  * The query tokens and the retained tokens of each visual chunk are each
    averaged into one representative feature vector.
  * Query/chunk similarity is the cosine of the two representative features
    (the retrieval equation of Sec. 3).
  * Only the top-k chunks by similarity (k is the retrieval budget "ur") are
    visible to the query tokens; the training mask of Eq. (4) instead keeps the
    chunks whose similarity reaches a threshold tau_q.  Both rules are
    supported: candidates are the chunks with s >= tau_q, of which the k
    largest are kept (tau_q = -inf gives plain top-k).
  * The query tokens then attend with softmax(Q K~^T / sqrt(d)) V~ over the
    keys and values of the retrieved chunks.

Readings taken where the paper is silent (each is also recorded in the design
notes):
  * A zero representative vector has no direction; its cosine with anything is
    taken as 0.
  * Equal scores: the earlier chunk (smaller index) ranks first.  The selected
    chunks are returned in stream order (ascending index), so the gathered
    keys keep their temporal order; softmax attention does not depend on key
    order.
  * Key set of query row i: the sink prefix, then the retrieved chunks in
    stream order, then the query/answer tokens themselves up to and including
    row i (causal).  With Lq query rows at the end of a tail of T tokens, row i
    sees tail tokens 0 .. T - Lq + i.  Lq = 1 is a decode step.
  * Grouped-query heads and 1/sqrt(d) as for the chunk prefill.

Test infrastructure only; shares no code with the HIP path.
"""
from __future__ import annotations

import math

import numpy as np

from .attention import default_scale, kv_head_of, softmax_attention


def token_mean(x: np.ndarray) -> np.ndarray:
    """Representative feature of a token sequence: the mean over tokens.

    x [L, dm] float64, L >= 1.  Returns [dm]."""
    x = np.asarray(x, dtype=np.float64)
    if x.shape[0] < 1:
        raise ValueError("the mean of zero tokens is undefined")
    return np.sum(x, axis=0) / x.shape[0]


def cosine_scores(q_feat: np.ndarray, chunk_feats: np.ndarray) -> np.ndarray:
    """s_i = <q, c_i> / (|q| |c_i|) for every chunk feature row c_i.

    q_feat [dm], chunk_feats [N, dm].  A zero vector on either side gives 0."""
    q = np.asarray(q_feat, dtype=np.float64)
    c = np.asarray(chunk_feats, dtype=np.float64)
    dots = c @ q
    denom = np.sqrt(np.sum(c * c, axis=1)) * math.sqrt(float(q @ q))
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(denom > 0, dots / np.where(denom > 0, denom, 1.0), 0.0)


def select_chunks(scores: np.ndarray, k: int, min_score: float = -math.inf) -> np.ndarray:
    """Indices of the k best chunks among those with score >= min_score.

    Ranking: larger score first, equal scores by smaller index.  Returns the
    selected indices in ascending order (stream order); fewer than k if fewer
    chunks qualify."""
    s = np.asarray(scores, dtype=np.float64)
    cand = [i for i in range(len(s)) if s[i] >= min_score]
    cand.sort(key=lambda i: (-s[i], i))
    return np.array(sorted(cand[:k]), dtype=np.int64)


def chunk_segments(selected: np.ndarray, chunk_start: np.ndarray, chunk_len: np.ndarray):
    """Store slot ranges (start, length) of the selected chunks, in the given order."""
    sel = np.asarray(selected, dtype=np.int64)
    return np.asarray(chunk_start, dtype=np.int64)[sel], np.asarray(chunk_len, dtype=np.int64)[sel]


def gathered_keys(store: np.ndarray, seg_start, seg_len, kv: int) -> np.ndarray:
    """Rows of the store listed by the segments, concatenated in segment order."""
    parts = [store[int(a):int(a) + int(n), kv] for a, n in zip(seg_start, seg_len)]
    if not parts:
        return np.zeros((0, store.shape[2]))
    return np.concatenate(parts, axis=0)


def gather_attention(q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len,
                     scale: float | None = None, heads=None):
    """Short-query attention over sink ++ retrieved store segments ++ causal tail.

    q [Lq, Hq, d]: the last Lq of T tail tokens; tail_k, tail_v [T, Hkv, d];
    sink_k, sink_v [S, Hkv, d]; store_k, store_v [cap, Hkv, d]; segments give
    store slot ranges [start, start + len).  All float64.
    Returns out [Lq, len(heads), d] and lse [len(heads), Lq] (natural log).
    """
    Lq, Hq, d = q.shape
    T, Hkv = tail_k.shape[0], tail_k.shape[1]
    if Lq > T:
        raise ValueError("the query rows are the last Lq of the T tail tokens")
    for a, n in zip(seg_start, seg_len):
        if a < 0 or n < 0 or a + n > store_k.shape[0]:
            raise ValueError(f"segment [{a}, {a + n}) outside the store")
    if scale is None:
        scale = default_scale(d)
    heads = np.arange(Hq) if heads is None else np.asarray(heads, dtype=np.int64)
    S = sink_k.shape[0]
    out = np.zeros((Lq, len(heads), d))
    lse = np.zeros((len(heads), Lq))
    for hi, h in enumerate(heads):
        kv = kv_head_of(int(h), Hq, Hkv)
        gk = gathered_keys(store_k, seg_start, seg_len, kv)
        gv = gathered_keys(store_v, seg_start, seg_len, kv)
        G = gk.shape[0]
        keys = np.concatenate([sink_k[:, kv], gk, tail_k[:, kv]], axis=0)
        vals = np.concatenate([sink_v[:, kv], gv, tail_v[:, kv]], axis=0)
        visible = np.ones((Lq, S + G + T), dtype=bool)
        tail_pos = np.arange(T)
        row_pos = T - Lq + np.arange(Lq)
        visible[:, S + G:] = tail_pos[None, :] <= row_pos[:, None]
        o, ls = softmax_attention(q[:, h], keys, vals, visible, scale)
        out[:, hi] = o
        lse[hi] = ls
    return out, lse
