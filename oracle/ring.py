"""Linear-history model of the ring-buffer visual KV cache (oracle side).

The paper bounds the visual cache each chunk can see (Sec. 3, "LLM
Prefilling and Decoding": the bound keeps the visible cache size fixed as
the stream grows).  The cache is realised as a ring of R token slots:
linear history position p lives in slot p mod R, so appending chunk
tokens x[0..C) after H history tokens writes slot (H + j) mod R for each j,
in order, later writes replacing earlier ones.  The W newest history tokens
are then read from slots (H - W + k) mod R, k = 0..W-1.

Rows are opaque (any dtype; the tests use bfloat16 bit patterns), so every
check on this model is bitwise.  Test infrastructure only.
"""
from __future__ import annotations

import numpy as np


class RingModel:
    def __init__(self, slots: int, row_shape=(), dtype=np.uint16):
        if slots <= 0:
            raise ValueError("ring needs at least one slot")
        self.slots = int(slots)
        self.buf = np.zeros((self.slots,) + tuple(row_shape), dtype=dtype)

    def append(self, chunk: np.ndarray, hist_len: int) -> int:
        """Write chunk[j] to slot (hist_len + j) mod R for j = 0..C-1 in order.

        Returns the new history length hist_len + C.
        """
        C = chunk.shape[0]
        for j in range(C):
            self.buf[(hist_len + j) % self.slots] = chunk[j]
        return hist_len + C

    def gather(self, hist_len: int, count: int) -> np.ndarray:
        """The `count` newest history tokens, oldest first, read through the slots."""
        if count > self.slots or count > hist_len:
            raise ValueError("requested tokens are not resident in the ring")
        return np.stack([self.buf[(hist_len - count + k) % self.slots] for k in range(count)]) \
            if count else self.buf[:0].copy()

    @classmethod
    def from_linear(cls, lin: np.ndarray, first_pos: int, slots: int) -> "RingModel":
        """Ring state after the tokens lin[0..n) (linear positions first_pos..) were appended."""
        r = cls(slots, lin.shape[1:], lin.dtype)
        r.append(lin, first_pos)
        return r
