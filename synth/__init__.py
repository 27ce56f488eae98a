"""Seeded synthetic inputs shared by the oracle-side tests and the HIP path.

This module only draws random numbers and rounds them to bfloat16 bit
patterns.  It contains none of the attention arithmetic: the oracle and the
HIP library each consume the arrays it returns on their own.

Workload shapes follow Qwen2.5-VL-3B/7B attention layers (post-RoPE Q/K/V,
grouped-query heads), which is what the streaming LLM prefill of the paper
(Sec. 3, "LLM Prefilling and Decoding") runs on.  Real video benchmarks are
not available, so Gaussian tensors stand in for the activations.

Draw order for one chunk is fixed: Q, K_chunk, V_chunk, sink_K, sink_V,
hist_K, hist_V.  Every tensor is drawn as float32 standard normal times a
scale, then rounded to bfloat16 with round-to-nearest-even.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "f32_to_bf16_bits",
    "ChunkShape",
    "ChunkInputs",
    "make_chunk_inputs",
    "ragged_chunk_lengths",
    "stream_chunk",
    "CONFIGS",
    "QueryShape",
    "QueryInputs",
    "make_query_inputs",
    "make_tokens",
    "QUERY_CONFIGS",
    "make_drop_frames",
    "DROP_CONFIGS",
]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even); return uint16 bits.

    Inputs are finite Gaussian draws, so no NaN/Inf handling is needed.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = (b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


@dataclass(frozen=True)
class ChunkShape:
    """Shape of one chunk-prefill attention call.

    hist_len is the linear count of visual tokens appended before this chunk;
    window is the number of most recent history tokens visible (-1: all).
    """
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    sink_len: int
    ring_slots: int
    hist_len: int
    window: int
    chunk_len: int

    @property
    def visible_window(self) -> int:
        if self.window < 0:
            return self.hist_len
        return min(self.window, self.hist_len)

    @property
    def hist_stored(self) -> int:
        """History positions that are still resident in the ring."""
        return min(self.hist_len, self.ring_slots)


@dataclass
class ChunkInputs:
    """bf16 bit patterns (uint16) for one chunk call.

    hist_k/hist_v hold linear history positions [hist_len - hist_stored,
    hist_len), oldest first.  Placing them into ring slots is the caller's job.
    """
    shape: ChunkShape
    q: np.ndarray          # [C, Hq, d]
    k_chunk: np.ndarray    # [C, Hkv, d]
    v_chunk: np.ndarray    # [C, Hkv, d]
    sink_k: np.ndarray     # [S, Hkv, d]
    sink_v: np.ndarray     # [S, Hkv, d]
    hist_k: np.ndarray     # [min(H, R), Hkv, d]
    hist_v: np.ndarray     # [min(H, R), Hkv, d]
    hist_first: int = field(default=0)   # linear position of hist_k[0]


def _draw(rng: np.random.Generator, shape, sigma: float) -> np.ndarray:
    if sigma == "U":      # uniform in [-1, 1)
        return f32_to_bf16_bits(rng.uniform(-1.0, 1.0, shape).astype(np.float32))
    return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(sigma))


def make_chunk_inputs(shape: ChunkShape, seed=0, family: str = "F1") -> ChunkInputs:
    """Draw all tensors of one chunk call.

    family "F1": Q, K, V ~ N(0,1)/sqrt(head_dim) (the literal workload recipe).
    family "F2": Q, K ~ 2*N(0,1), V ~ N(0,1): logits of standard deviation 4
                 and O(1) outputs, used for the binding parity tolerance.
    family "F2U": Q, K as in F2, V uniform in [-1, 1): every output lies in
                 [-1, 1], the literal reading of "O(1)-scaled outputs".
    """
    d = shape.head_dim
    if family == "F1":
        sq = sk = sv = 1.0 / np.sqrt(d)
    elif family == "F2":
        sq, sk, sv = 2.0, 2.0, 1.0
    elif family == "F2U":
        sq, sk, sv = 2.0, 2.0, "U"
    else:
        raise ValueError(f"unknown input family {family!r}")
    rng = np.random.Generator(np.random.PCG64(seed))
    C, Hq, Hkv, S = shape.chunk_len, shape.num_q_heads, shape.num_kv_heads, shape.sink_len
    n_hist = shape.hist_stored
    q = _draw(rng, (C, Hq, d), sq)
    kc = _draw(rng, (C, Hkv, d), sk)
    vc = _draw(rng, (C, Hkv, d), sv)
    sk_ = _draw(rng, (S, Hkv, d), sk)
    sv_ = _draw(rng, (S, Hkv, d), sv)
    hk = _draw(rng, (n_hist, Hkv, d), sk)
    hv = _draw(rng, (n_hist, Hkv, d), sv)
    return ChunkInputs(shape, q, kc, vc, sk_, sv_, hk, hv, hist_first=shape.hist_len - n_hist)


def ragged_chunk_lengths(n_chunks: int = 64, lo: int = 256, hi: int = 1024, seed: int = 0) -> np.ndarray:
    """Retained-token counts per chunk, uniform in [lo, hi] (token-dropping output)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(lo, hi + 1, n_chunks)


def stream_chunk(t: int, chunk_len: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                 seed: int = 0, family: str = "F1"):
    """Q/K/V bits of streaming chunk t: drawn from PCG64([seed, t]) in order Q, K, V."""
    d = head_dim
    if family == "F1":
        sq = sk = sv = 1.0 / np.sqrt(d)
    else:
        sq, sk, sv = 2.0, 2.0, 1.0
    rng = np.random.Generator(np.random.PCG64([seed, t]))
    q = _draw(rng, (chunk_len, num_q_heads, d), sq)
    k = _draw(rng, (chunk_len, num_kv_heads, d), sk)
    v = _draw(rng, (chunk_len, num_kv_heads, d), sv)
    return q, k, v


def stream_sink(sink_len: int, num_kv_heads: int, head_dim: int, seed: int = 0, family: str = "F1"):
    """Sink K/V bits for a stream, drawn from PCG64([seed, 1 << 20])."""
    d = head_dim
    sk, sv = (1.0 / np.sqrt(d),) * 2 if family == "F1" else (2.0, 1.0)
    rng = np.random.Generator(np.random.PCG64([seed, 1 << 20]))
    return _draw(rng, (sink_len, num_kv_heads, d), sk), _draw(rng, (sink_len, num_kv_heads, d), sv)


# Workload shapes (one attention layer each).  The ring holds exactly W slots.
CONFIGS = {
    # tiny: 2/1 heads, d 64, sink 16, W = R = 256, chunk 64; ring write pointer at 200.
    "tiny": ChunkShape(2, 1, 64, 16, 256, 456, 256, 64),
    "tiny_partial": ChunkShape(2, 1, 64, 16, 256, 200, 256, 64),
    # Qwen2.5-VL-3B layer: 16/2 heads, d 128, sink 64, W = R = 8192, chunk 1024.
    "3b": ChunkShape(16, 2, 128, 64, 8192, 8192, 8192, 1024),
    "3b_wrap": ChunkShape(16, 2, 128, 64, 8192, 5 * 8192 + 777, 8192, 1024),
    # Qwen2.5-VL-7B layer: 28/4 heads, d 128, sink 64, W = R = 16384, chunk 2048.
    "7b": ChunkShape(28, 4, 128, 64, 16384, 16384, 16384, 2048),
    "7b_wrap": ChunkShape(28, 4, 128, 64, 16384, 5 * 16384 + 777, 16384, 2048),
    # full history (65536 tokens) vs bounded W = 8192 at 3B heads, chunk 2048.
    "full": ChunkShape(16, 2, 128, 64, 65536, 65536, -1, 2048),
    "full_bounded": ChunkShape(16, 2, 128, 64, 65536, 65536, 8192, 2048),
}


# ---------------------------------------------------------------------------
# Query-side retrieval workloads: a store of past chunks (linear history of
# K/V), one representative feature per chunk, and a short query.
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class QueryShape:
    """Shape of one query-side call (retrieval + attention over retrieved chunks).

    feat_dim is the LLM hidden size of the representative features; the store
    holds num_chunks chunks of ragged length in [chunk_lo, chunk_hi], stored one
    after another; q_len query rows are the last of tail_len tail tokens."""
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    sink_len: int
    feat_dim: int
    num_chunks: int
    chunk_lo: int
    chunk_hi: int
    q_len: int
    tail_len: int
    top_k: int


@dataclass
class QueryInputs:
    shape: QueryShape
    chunk_len: np.ndarray      # [N] int64 retained tokens per chunk
    chunk_start: np.ndarray    # [N] int64 first store slot of each chunk
    chunk_feat: np.ndarray     # [N, dm] float32 representative features
    query_x: np.ndarray        # [Lq, dm] bf16 bits: query token embeddings
    q: np.ndarray              # [Lq, Hq, d] bf16 bits
    tail_k: np.ndarray         # [T, Hkv, d]
    tail_v: np.ndarray
    sink_k: np.ndarray         # [S, Hkv, d]
    sink_v: np.ndarray
    seed: int = 0
    family: str = "F1"

    @property
    def store_len(self) -> int:
        return int(self.chunk_start[-1] + self.chunk_len[-1]) if len(self.chunk_len) else 0

    def chunk_kv(self, i: int):
        """K/V bits of stored chunk i, drawn from PCG64([seed, 3, i]) in order K, V."""
        sh = self.shape
        _, sk, sv = _family_sigmas(self.family, sh.head_dim)
        rng = np.random.Generator(np.random.PCG64([self.seed, 3, i]))
        n = int(self.chunk_len[i])
        return (_draw(rng, (n, sh.num_kv_heads, sh.head_dim), sk),
                _draw(rng, (n, sh.num_kv_heads, sh.head_dim), sv))

    def store_kv(self):
        """The whole store [store_len, Hkv, d] (K, V), chunk after chunk."""
        ks, vs = zip(*(self.chunk_kv(i) for i in range(len(self.chunk_len))))
        return np.concatenate(ks, axis=0), np.concatenate(vs, axis=0)


def _family_sigmas(family: str, d: int):
    if family == "F2U":
        return 2.0, 2.0, "U"
    if family == "F1":
        return (1.0 / np.sqrt(d),) * 3
    if family == "F2":
        return 2.0, 2.0, 1.0
    raise ValueError(f"unknown input family {family!r}")


def make_query_inputs(shape: QueryShape, seed=0, family: str = "F1", num_topics: int = 16,
                      query_seed: int = 0) -> QueryInputs:
    """Draw a query-side workload.

    Features follow a topic mixture so that similarities spread out: topic
    vectors t_j ~ N(0,1); chunk i gets a topic and feature t + 0.75 N(0,1);
    the query tokens are t_q + N(0,1) for one topic t_q.  Streams:
    PCG64([seed, 1]) lengths and features, PCG64([seed, 2]) query tokens,
    q and tail (PCG64([seed, 2, query_seed]) for query_seed > 0: another
    query over the same store), PCG64([seed, 3, i]) chunk i's K/V,
    PCG64([seed, 4]) sink."""
    sh = shape
    sq, sk, sv = _family_sigmas(family, sh.head_dim)
    rng = np.random.Generator(np.random.PCG64([seed, 1]))
    lens = rng.integers(sh.chunk_lo, sh.chunk_hi + 1, sh.num_chunks).astype(np.int64)
    start = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    topics = rng.standard_normal((num_topics, sh.feat_dim), dtype=np.float32)
    which = rng.integers(0, num_topics, sh.num_chunks)
    feat = (topics[which] + np.float32(0.75) * rng.standard_normal((sh.num_chunks, sh.feat_dim),
                                                                   dtype=np.float32)).astype(np.float32)
    rq = np.random.Generator(np.random.PCG64([seed, 2] if query_seed == 0 else [seed, 2, query_seed]))
    qt = int(rq.integers(0, num_topics))
    query_x = f32_to_bf16_bits(topics[qt][None, :] + rq.standard_normal((sh.q_len, sh.feat_dim), dtype=np.float32))
    q = _draw(rq, (sh.q_len, sh.num_q_heads, sh.head_dim), sq)
    tk = _draw(rq, (sh.tail_len, sh.num_kv_heads, sh.head_dim), sk)
    tv = _draw(rq, (sh.tail_len, sh.num_kv_heads, sh.head_dim), sv)
    rs = np.random.Generator(np.random.PCG64([seed, 4]))
    snk = _draw(rs, (sh.sink_len, sh.num_kv_heads, sh.head_dim), sk)
    snv = _draw(rs, (sh.sink_len, sh.num_kv_heads, sh.head_dim), sv)
    return QueryInputs(sh, lens, start, feat, query_x, q, tk, tv, snk, snv, seed=seed, family=family)


def make_tokens(n_tokens: int, feat_dim: int, seed=0, offset: float = 0.0) -> np.ndarray:
    """bf16 bits [n_tokens, feat_dim] of N(offset, 1) token embeddings, PCG64([seed, 5])."""
    rng = np.random.Generator(np.random.PCG64([seed, 5]))
    return f32_to_bf16_bits(np.float32(offset) + rng.standard_normal((n_tokens, feat_dim), dtype=np.float32))


# Query-side shapes.  Store chunks have 256..1024 retained tokens (25-100 %
# of a 1024-token chunk); the query is 32 tokens; ur = 32 retrieved chunks.
QUERY_CONFIGS = {
    "q_tiny": QueryShape(2, 1, 64, 8, 256, 12, 5, 40, 4, 6, 3),
    "q_small": QueryShape(8, 2, 128, 16, 512, 40, 16, 200, 16, 16, 8),
    "q_gqa7": QueryShape(14, 2, 128, 4, 384, 30, 1, 300, 9, 21, 7),
    "q_7b": QueryShape(28, 4, 128, 64, 3584, 256, 256, 1024, 32, 32, 32),
    "q_3b": QueryShape(16, 2, 128, 64, 2048, 256, 256, 1024, 32, 32, 32),
}


# ---------------------------------------------------------------------------
# Temporal token dropping: projected visual tokens of consecutive frames.
# ---------------------------------------------------------------------------

def make_drop_frames(num_chunks: int, frames_per_chunk: int, tokens_per_frame: int, feat_dim: int,
                     static_frac: float = 0.5, noise: float = 0.15, seed: int = 0) -> np.ndarray:
    """bf16 bits [B, c, n_f, dm] of projected tokens with static and moving regions.

    Every position gets a base vector ~ N(0,1).  A static position (a fraction
    static_frac, fixed per position for the whole batch) shows the base plus
    noise * N(0,1) in every frame, so its frames are nearly parallel (cosine
    about 1 / (1 + noise^2)); a moving position draws a fresh N(0,1) vector
    per frame (cosine about 0).  A few positions use noise levels spread
    around the usual thresholds so that similarities fall close to them.
    Drawn from PCG64([seed, 6])."""
    rng = np.random.Generator(np.random.PCG64([seed, 6]))
    B, c, n_f, dm = num_chunks, frames_per_chunk, tokens_per_frame, feat_dim
    static = rng.random(n_f) < static_frac
    level = np.full(n_f, noise, dtype=np.float32)
    near = rng.random(n_f) < 0.1
    level[near] = rng.uniform(0.2, 0.6, int(near.sum())).astype(np.float32)
    out = np.empty((B, c, n_f, dm), dtype=np.uint16)
    base = rng.standard_normal((n_f, dm), dtype=np.float32)
    for b in range(B):
        for f in range(c):
            fresh = rng.standard_normal((n_f, dm), dtype=np.float32)
            x = np.where(static[:, None], base + level[:, None] * fresh, fresh)
            out[b, f] = f32_to_bf16_bits(x)
        if rng.random() < 0.3:                     # the scene changes between chunks now and then
            base = rng.standard_normal((n_f, dm), dtype=np.float32)
    return out


# (num_chunks, frames per chunk, tokens per frame, feature dim): Qwen2.5-VL
# merges 2x2 patches of 14 px, so a 448x448 frame gives 16 x 16 = 256 tokens;
# 4 frames per chunk give the 1024-token chunks of the streaming workload.
DROP_CONFIGS = {
    "tiny": (3, 4, 24, 64),
    "c2": (2, 2, 40, 128),
    "c1": (6, 1, 32, 96),
    "c8": (1, 8, 50, 256),
    "7b": (16, 4, 256, 3584),
    "3b": (16, 4, 256, 2048),
}
