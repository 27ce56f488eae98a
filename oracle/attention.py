"""Exact bounded chunk-prefill attention in float64 (oracle side).

Definition followed (paper, Sec. 3, "LLM Prefilling and Decoding"): for the
current visual chunk, Attn = softmax(Q K_hat^T / sqrt(d)) V_hat, where K_hat /
V_hat are the keys and values the chunk may see.  The vision rows of the
additive mask of Eq. (4) say which keys those are: recent visual history and
the current chunk, everything else masked with -inf.

Readings taken where the paper is silent or loose:
  * Window unit: the visible history is the W most recent history *tokens*
    (the token-granular "Nearest-K" context of the nearest-visual-context
    table), not whole chunks; W < 0 means the full history.
  * The visible window is Wv = min(W, H) tokens, H = tokens appended before
    the chunk; the current chunk is not counted in W.
  * A sink prefix of S tokens (system/text tokens) precedes all visual tokens,
    is always visible and is never evicted.  The paper does not mention it.
  * Inside the chunk the mask is causal: row i sees chunk keys 0..i (decoder
    LLM).  Eq. (4) read literally would expose the whole chunk to itself.
  * d in the 1/sqrt(d) scale is the head dimension.
  * Grouped-query attention: query head h reads KV head floor(h / g), with
    g = Hq / Hkv (contiguous head groups).

Two independent formulations are provided and cross-checked by the tests:
a blocked dense one (logits for a block of rows against all keys, boolean
mask from indices, two-pass softmax) and a per-row loop that walks the
visible keys one by one.  Test infrastructure only.
"""
from __future__ import annotations

import math

import numpy as np


def default_scale(head_dim: int) -> float:
    """Softmax temperature 1/sqrt(d), d = head dimension."""
    return 1.0 / math.sqrt(head_dim)


def visible_window(hist_len: int, window: int) -> int:
    """Number of history tokens visible to the chunk: min(W, H), or H if W < 0."""
    if window < 0:
        return hist_len
    return min(window, hist_len)


def kv_head_of(h: int, num_q_heads: int, num_kv_heads: int) -> int:
    """KV head read by query head h under grouped-query attention."""
    g = num_q_heads // num_kv_heads
    return h // g


def chunk_causal_mask(rows: np.ndarray, chunk_len: int) -> np.ndarray:
    """Boolean [len(rows), C]: chunk key j is visible to chunk row i iff j <= i."""
    j = np.arange(chunk_len)
    return j[None, :] <= np.asarray(rows)[:, None]


def softmax_attention(q: np.ndarray, keys: np.ndarray, vals: np.ndarray,
                      visible: np.ndarray, scale: float):
    """Masked softmax attention for a block of rows, float64.

    q [n, d], keys [L, d], vals [L, dv], visible [n, L] boolean.
    Returns (out [n, dv], lse [n]) with lse the natural-log sum of
    exp(scale * q.k) over visible keys.  A row with no visible key gets
    out = 0 and lse = -inf.
    """
    z = (q @ keys.T) * scale
    z = np.where(visible, z, -np.inf)
    m = np.max(z, axis=1, keepdims=True)
    m_safe = np.where(np.isfinite(m), m, 0.0)
    p = np.exp(z - m_safe)
    l = np.sum(p, axis=1, keepdims=True)
    with np.errstate(invalid="ignore", divide="ignore"):
        out = np.where(l > 0, (p @ vals) / np.where(l > 0, l, 1.0), 0.0)
        lse = np.where(l[:, 0] > 0, m_safe[:, 0] + np.log(np.where(l[:, 0] > 0, l[:, 0], 1.0)), -np.inf)
    return out, lse


def _check_shapes(q, k_chunk, v_chunk, sink_k, sink_v, hist_k, hist_v, hist_len, window):
    C, Hq, d = q.shape
    Hkv = k_chunk.shape[1]
    if Hq % Hkv:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    wv = visible_window(hist_len, window)
    if hist_k.shape[0] < wv:
        raise ValueError(f"history holds {hist_k.shape[0]} tokens, window needs {wv}")
    return C, Hq, Hkv, d, wv


def chunk_prefill_attention(q, k_chunk, v_chunk, sink_k, sink_v, hist_k, hist_v,
                            hist_len: int, window: int, scale: float | None = None,
                            rows=None, heads=None, block_rows: int = 256, bidirectional: bool = False):
    """Bounded chunk-prefill attention, blocked dense form.

    q [C, Hq, d]; k_chunk, v_chunk [C, Hkv, d]; sink_k, sink_v [S, Hkv, d];
    hist_k, hist_v [n, Hkv, d]: the last n >= Wv history tokens in linear
    order (position hist_len - n first).  All float64.
    rows / heads select which chunk rows and query heads to compute.
    bidirectional: every row sees the whole chunk (Eq. (4) read literally:
    a vision token sees every token of the chunks in its window, its own
    chunk included) instead of chunk keys 0..i.
    Returns out [len(rows), len(heads), d] and lse [len(heads), len(rows)].
    """
    C, Hq, Hkv, d, wv = _check_shapes(q, k_chunk, v_chunk, sink_k, sink_v, hist_k, hist_v,
                                      hist_len, window)
    if scale is None:
        scale = default_scale(d)
    rows = np.arange(C) if rows is None else np.asarray(rows, dtype=np.int64)
    heads = np.arange(Hq) if heads is None else np.asarray(heads, dtype=np.int64)
    S = sink_k.shape[0]
    n = hist_k.shape[0]
    out = np.zeros((len(rows), len(heads), d))
    lse = np.zeros((len(heads), len(rows)))
    for hi, h in enumerate(heads):
        kv = kv_head_of(int(h), Hq, Hkv)
        keys = np.concatenate([sink_k[:, kv], hist_k[n - wv:n, kv], k_chunk[:, kv]], axis=0)
        vals = np.concatenate([sink_v[:, kv], hist_v[n - wv:n, kv], v_chunk[:, kv]], axis=0)
        for b0 in range(0, len(rows), block_rows):
            rb = rows[b0:b0 + block_rows]
            visible = np.ones((len(rb), S + wv + C), dtype=bool)
            if not bidirectional:
                visible[:, S + wv:] = chunk_causal_mask(rb, C)
            o, ls = softmax_attention(q[rb, h], keys, vals, visible, scale)
            out[b0:b0 + len(rb), hi] = o
            lse[hi, b0:b0 + len(rb)] = ls
    return out, lse


def chunk_prefill_attention_rowloop(q, k_chunk, v_chunk, sink_k, sink_v, hist_k, hist_v,
                                    hist_len: int, window: int, scale: float | None = None):
    """Same result, one row at a time: list the visible keys, then softmax.

    Walks the key set explicitly (sink tokens, then the Wv newest history
    tokens, then chunk tokens 0..i) and accumulates exp(z - max) in plain
    Python floats.  Only for tiny inputs.
    """
    C, Hq, d = q.shape
    Hkv = k_chunk.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    S = sink_k.shape[0]
    n = hist_k.shape[0]
    first = 0 if window < 0 else max(0, hist_len - window)   # oldest visible position
    if first < hist_len - n:
        raise ValueError("history does not reach back to the window start")
    out = np.zeros((C, Hq, d))
    lse = np.zeros((Hq, C))
    for h in range(Hq):
        kv = (h * Hkv) // Hq          # contiguous groups of Hq / Hkv query heads
        for i in range(C):
            ks, vs = [], []
            for s in range(S):
                ks.append(sink_k[s, kv]); vs.append(sink_v[s, kv])
            for p in range(first, hist_len):
                idx = p - (hist_len - n)
                ks.append(hist_k[idx, kv]); vs.append(hist_v[idx, kv])
            for j in range(i + 1):
                ks.append(k_chunk[j, kv]); vs.append(v_chunk[j, kv])
            z = [scale * math.fsum(float(a) * float(b) for a, b in zip(q[i, h], kk)) for kk in ks]
            m = max(z)
            w = [math.exp(zz - m) for zz in z]
            l = math.fsum(w)
            for c in range(d):
                out[i, h, c] = math.fsum(ww * float(vv[c]) for ww, vv in zip(w, vs)) / l
            lse[h, i] = m + math.log(l)
    return out, lse


def acn_window(chunk_starts, t: int, acn: int) -> int:
    """History tokens visible to chunk t under the chunk-granular window.

    The vision rows of Eq. (4) see the chunks t-acn .. t (the staircase band);
    with chunk t starting at linear position chunk_starts[t] (history tokens
    appended before it), the visible history is chunks max(0, t-acn) .. t-1:
    chunk_starts[t] - chunk_starts[max(0, t - acn)] tokens.  acn < 0 means the
    whole history.  The window then goes to chunk_prefill_attention."""
    starts = np.asarray(chunk_starts, dtype=np.int64)
    if acn < 0:
        return int(starts[t])
    return int(starts[t] - starts[max(0, t - acn)])
