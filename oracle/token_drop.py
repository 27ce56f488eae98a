"""Chunk-level temporal token dropping, float64 (oracle side).

Definition followed (paper, Sec. 3, "Token Dropping", temporal compression):
for every spatial position p of a chunk of c frames, the cosine similarity of
the projected tokens of every frame pair i < j is taken (the pairwise
similarity equation); position p is dropped when all of them exceed the
threshold tau (the drop equation).  The first frame of every chunk is always
kept as an anchor.  With c = 1 the rule degenerates to frame-level dropping:
a frame's token is dropped when its similarity to the same position of the
previous frame exceeds tau, with no anchor.

Readings taken where the paper is silent:
  * A dropped position loses its tokens in frames 2..c; frame 1's token
    stays (the anchor).  A position that is not dropped keeps all c tokens.
  * Retained tokens keep stream order: chunk by chunk, frame by frame, and
    by position within a frame.
  * A zero vector has no direction; its cosine with anything is taken as 0.
  * c = 1: the first frame of a batch is compared with `prev` (the frame
    before it in the stream) when given, and kept whole otherwise; every
    later frame is compared with the frame before it.
  * "Exceed" is strict: a similarity equal to tau does not drop.

Test infrastructure only; shares no code with the HIP path.
"""
from __future__ import annotations

import numpy as np

NO_COMPARISON = -2.0   # similarity reported for a token nothing is compared with (kept)


def _cos(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Row-wise cosine of two [n, dm] arrays; 0 where either row is zero."""
    dots = np.sum(a * b, axis=1)
    den = np.sqrt(np.sum(a * a, axis=1)) * np.sqrt(np.sum(b * b, axis=1))
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(den > 0, dots / np.where(den > 0, den, 1.0), 0.0)


def temporal_drop(z: np.ndarray, tau: float, prev: np.ndarray | None = None):
    """Temporal token dropping over a batch of chunks.

    z [B, c, n_f, dm] float64: B consecutive chunks of c frames.
    prev [n_f, dm]: the frame before the batch (c = 1 only), or None.
    Returns (keep [B, n_f] bool, sim [B, n_f], index [n_keep] int64) where
    keep says whether position p survives (frames 2..c for c > 1, the frame
    itself for c = 1), sim is the smallest pairwise similarity of the
    position (the similarity to the previous frame for c = 1;
    NO_COMPARISON when there is nothing to compare with), and index lists
    the retained tokens in stream order as flat indices (b * c + f) * n_f + p
    into z viewed as [B * c * n_f, dm].
    """
    z = np.asarray(z, dtype=np.float64)
    B, c, n_f, _ = z.shape
    keep = np.ones((B, n_f), dtype=bool)
    sim = np.full((B, n_f), NO_COMPARISON)
    for b in range(B):
        if c > 1:
            drop = np.ones(n_f, dtype=bool)
            smin = np.full(n_f, np.inf)
            for i in range(c):
                for j in range(i + 1, c):
                    s_ij = _cos(z[b, i], z[b, j])
                    drop &= s_ij > tau              # the conjunction over all pairs i < j
                    smin = np.minimum(smin, s_ij)
            sim[b] = smin
            keep[b] = ~drop
        else:
            before = z[b - 1, 0] if b > 0 else prev
            if before is not None:
                s = _cos(z[b, 0], np.asarray(before, dtype=np.float64))
                sim[b] = s
                keep[b] = ~(s > tau)
    return keep, sim, retained_index(keep, c)


def retained_index(keep: np.ndarray, c: int) -> np.ndarray:
    """Flat source rows of the retained tokens, in stream order, for the
    position decisions `keep` [B, n_f] of chunks of c frames: every token of
    the anchor frame (c > 1), and the tokens of kept positions in the other
    frames (all frames when c = 1)."""
    B, n_f = keep.shape
    index = []
    for b in range(B):
        for f in range(c):
            for p in range(n_f):
                if (c > 1 and f == 0) or keep[b, p]:
                    index.append((b * c + f) * n_f + p)
    return np.asarray(index, dtype=np.int64)


def gather_tokens(z: np.ndarray, index: np.ndarray) -> np.ndarray:
    """The retained tokens, [n_keep, dm], in the order of `index`."""
    B, c, n_f, dm = z.shape
    return np.asarray(z).reshape(B * c * n_f, dm)[np.asarray(index, dtype=np.int64)]
