"""Helpers shared by the tests: oracle inputs from synthetic bf16 bits."""
from __future__ import annotations

import numpy as np

import oracle
from synth import ChunkInputs


def to_f64(inp: ChunkInputs):
    """Oracle view of one chunk call: float64 arrays widened from the bf16 bits."""
    w = oracle.bf16_bits_to_f64
    return dict(q=w(inp.q), k_chunk=w(inp.k_chunk), v_chunk=w(inp.v_chunk),
                sink_k=w(inp.sink_k), sink_v=w(inp.sink_v),
                hist_k=w(inp.hist_k), hist_v=w(inp.hist_v),
                hist_len=inp.shape.hist_len, window=inp.shape.window)


def ring_from_inputs(inp: ChunkInputs):
    """Ring K/V slot arrays (bf16 bits) holding the stored history of `inp`."""
    sh = inp.shape
    rk = oracle.RingModel.from_linear(inp.hist_k, inp.hist_first, sh.ring_slots).buf if sh.ring_slots else \
        np.zeros((0, sh.num_kv_heads, sh.head_dim), np.uint16)
    rv = oracle.RingModel.from_linear(inp.hist_v, inp.hist_first, sh.ring_slots).buf if sh.ring_slots else \
        np.zeros((0, sh.num_kv_heads, sh.head_dim), np.uint16)
    return rk, rv
