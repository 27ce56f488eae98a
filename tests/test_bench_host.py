"""bench.py's algorithmic counts, on the CPU: the flop count a chunk call is
priced at (4 d flops per visible (query row, key) pair per query head,
masked pairs excluded) against a brute-force count of the visible pairs
from the oracle's visibility rules, and the per-layer figures of the 3B, 7B
and full-history workloads."""
import numpy as np
import pytest

import bench
import oracle
from oracle.attention import chunk_causal_mask


@pytest.mark.parametrize("C,S,H,W", [(64, 16, 456, 256), (64, 16, 200, 256), (300, 5, 1333, 600),
                                     (1, 64, 5000, 1000), (150, 0, 0, 0), (77, 7, 400, -1)])
def test_attn_flops_counts_the_visible_pairs(C, S, H, W):
    Wv = oracle.visible_window(H, W)
    pairs = 0
    for i in range(C):                                   # row by row: sink, window, chunk keys 0..i
        pairs += S + Wv + int(chunk_causal_mask(np.array([i]), C).sum())
    assert bench.attn_flops(C, S, Wv, 3, 64) == 4 * 3 * 64 * pairs
    rows = np.array([0, C // 2, C - 1])
    sub = sum(S + Wv + i + 1 for i in rows)
    assert bench.attn_flops(C, S, Wv, 3, 64, rows=rows) == 4 * 3 * 64 * sub


@pytest.mark.parametrize("name,flops", [("3b", 7.356e10), ("7b", 5.130e11), ("full", 1.118e12),
                                        ("full_bounded", 1.557e11)])
def test_workload_flops(name, flops):
    sh = bench.workload_shape(name)
    f = bench.attn_flops(sh.chunk_len, sh.sink_len, sh.visible_window, sh.num_q_heads, sh.head_dim)
    assert f == pytest.approx(flops, rel=5e-4)
    # closed form: 4 Hq d [C (S + Wv) + C (C + 1) / 2]
    C = sh.chunk_len
    assert f == 4 * sh.num_q_heads * sh.head_dim * (C * (sh.sink_len + sh.visible_window) + C * (C + 1) // 2)
