"""Pins of the query-side retrieval oracle against library routines, closed
forms, brute force and invariants (paper, Sec. 3, query-time decoding; query
rows of Eq. (4))."""
from __future__ import annotations

import dataclasses
import itertools
import math
import statistics

import numpy as np
import pytest
import torch
from scipy.spatial.distance import cdist

import oracle
from oracle import retrieval as R
from synth import QUERY_CONFIGS, make_query_inputs, make_tokens, CONFIGS, make_chunk_inputs
from tests._util import to_f64


def f64(bits):
    return oracle.bf16_bits_to_f64(bits)


# ---------------------------------------------------------------- token mean

def test_mean_of_constant_rows_is_the_constant():
    x = np.tile(np.linspace(-3, 5, 17), (9, 1))
    assert np.array_equal(R.token_mean(x), x[0])


def test_mean_of_arithmetic_sequence_closed_form():
    L = 101
    x = np.arange(L, dtype=np.float64)[:, None] * np.array([1.0, -2.0, 0.5])[None, :] + 7.0
    np.testing.assert_allclose(R.token_mean(x), 7.0 + (L - 1) / 2 * np.array([1.0, -2.0, 0.5]), rtol=0, atol=1e-12)


def test_mean_matches_statistics_fmean():
    x = f64(make_tokens(37, 64, seed=3))
    ref = np.array([statistics.fmean(x[:, j]) for j in range(x.shape[1])])
    np.testing.assert_allclose(R.token_mean(x), ref, rtol=0, atol=1e-14)


def test_mean_of_no_tokens_is_an_error():
    with pytest.raises(ValueError):
        R.token_mean(np.zeros((0, 4)))


# ---------------------------------------------------------------- cosine

def test_cosine_matches_scipy_cdist():
    rng = np.random.default_rng(0)
    q = rng.standard_normal(48)
    c = rng.standard_normal((30, 48))
    ref = 1.0 - cdist(q[None, :], c, metric="cosine")[0]
    np.testing.assert_allclose(R.cosine_scores(q, c), ref, rtol=0, atol=1e-13)


def test_cosine_special_values():
    e = np.eye(5)
    q = np.array([0.0, 3.0, 0.0, 0.0, 0.0])
    s = R.cosine_scores(q, np.vstack([e, -2 * q, 5 * q, np.zeros(5)]))
    np.testing.assert_allclose(s, [0, 1, 0, 0, 0, -1, 1, 0], atol=1e-15)


def test_cosine_scale_invariance_and_sign():
    rng = np.random.default_rng(1)
    q = rng.standard_normal(16)
    c = rng.standard_normal((7, 16))
    s = R.cosine_scores(q, c)
    np.testing.assert_allclose(R.cosine_scores(4.5 * q, c * np.arange(1, 8)[:, None]), s, atol=1e-14)
    np.testing.assert_allclose(R.cosine_scores(-q, c), -s, atol=1e-15)
    assert np.all(np.abs(s) <= 1 + 1e-15)


def test_zero_query_scores_zero():
    assert np.all(R.cosine_scores(np.zeros(8), np.ones((3, 8))) == 0)


# ---------------------------------------------------------------- selection

def _brute_force_select(s, k, tau=-math.inf):
    """The unique k-subset (or all candidates) such that every member outranks
    every non-member: a higher score, or an equal score and a smaller index."""
    cand = [i for i in range(len(s)) if s[i] >= tau]
    if len(cand) <= k:
        return sorted(cand)
    found = []
    for sub in itertools.combinations(cand, k):
        rest = [j for j in cand if j not in sub]
        if all((s[a] > s[b]) or (s[a] == s[b] and a < b) for a in sub for b in rest):
            found.append(sorted(sub))
    assert len(found) == 1
    return found[0]


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("k", [1, 3, 5])
def test_select_matches_brute_force_with_ties(seed, k):
    rng = np.random.default_rng(seed)
    s = np.round(rng.uniform(-1, 1, 9), 1)          # coarse values force ties
    assert list(R.select_chunks(s, k)) == _brute_force_select(s, k)


@pytest.mark.parametrize("tau", [-0.5, 0.0, 0.3, 0.95])
def test_select_threshold_matches_brute_force(tau):
    rng = np.random.default_rng(7)
    s = np.round(rng.uniform(-1, 1, 10), 1)
    got = list(R.select_chunks(s, 4, tau))
    assert got == _brute_force_select(s, 4, tau)
    assert all(s[i] >= tau for i in got)


def test_select_closed_forms():
    s = np.linspace(1, -1, 12)                       # strictly decreasing in index
    assert list(R.select_chunks(s, 5)) == [0, 1, 2, 3, 4]
    assert list(R.select_chunks(np.zeros(6), 4)) == [0, 1, 2, 3]    # all tied: earliest
    assert list(R.select_chunks(s, 50)) == list(range(12))          # k > N keeps all
    assert list(R.select_chunks(s, 0)) == []


def test_segments_follow_the_chunk_table():
    st, ln = R.chunk_segments(np.array([4, 1]), np.array([0, 10, 25, 40, 70]), np.array([10, 15, 15, 30, 9]))
    assert list(st) == [70, 10] and list(ln) == [9, 15]


# ---------------------------------------------------------------- gathered attention

def _sdpa_reference(qi, seg_start, seg_len, heads=None):
    """torch scaled_dot_product_attention in float64 over keys listed slot by slot."""
    sh = qi.shape
    sk, sv = f64(qi.sink_k), f64(qi.sink_v)
    stk, stv = (f64(x) for x in qi.store_kv())
    tk, tv, q = f64(qi.tail_k), f64(qi.tail_v), f64(qi.q)
    g = sh.num_q_heads // sh.num_kv_heads
    slots = [p for a, n in zip(seg_start, seg_len) for p in range(int(a), int(a) + int(n))]
    T, Lq = sh.tail_len, sh.q_len
    outs, lses = [], []
    for h in range(sh.num_q_heads) if heads is None else heads:
        kv = h // g
        keys = np.concatenate([sk[:, kv], stk[slots, kv].reshape(-1, sh.head_dim), tk[:, kv]])
        vals = np.concatenate([sv[:, kv], stv[slots, kv].reshape(-1, sh.head_dim), tv[:, kv]])
        n_fixed = sh.sink_len + len(slots)
        mask = np.zeros((Lq, keys.shape[0]), dtype=bool)
        mask[:, :n_fixed] = True
        for i in range(Lq):
            mask[i, n_fixed:n_fixed + T - Lq + i + 1] = True
        o = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q[:, h])[None], torch.from_numpy(keys)[None], torch.from_numpy(vals)[None],
            attn_mask=torch.from_numpy(mask)[None])[0].numpy()
        z = (q[:, h] @ keys.T) / math.sqrt(sh.head_dim)
        lse = torch.logsumexp(torch.from_numpy(np.where(mask, z, -np.inf)), dim=1).numpy()
        outs.append(o)
        lses.append(lse)
    return np.stack(outs, axis=1), np.stack(lses)


def _call(qi, seg_start, seg_len, heads=None):
    stk, stv = (f64(x) for x in qi.store_kv())
    return R.gather_attention(f64(qi.q), f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k), f64(qi.sink_v),
                              stk, stv, seg_start, seg_len, heads=heads)


@pytest.mark.parametrize("name", ["q_tiny", "q_small", "q_gqa7"])
def test_gather_attention_matches_torch_sdpa(name):
    qi = make_query_inputs(QUERY_CONFIGS[name], seed=1, family="F2")
    sel = R.select_chunks(np.arange(qi.shape.num_chunks)[::-1] % 5, qi.shape.top_k)
    st, ln = R.chunk_segments(sel, qi.chunk_start, qi.chunk_len)
    out, lse = _call(qi, st, ln)
    ref_o, ref_l = _sdpa_reference(qi, st, ln)
    np.testing.assert_allclose(out, ref_o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, ref_l, rtol=0, atol=1e-12)


def test_gather_attention_segment_order_does_not_matter():
    qi = make_query_inputs(QUERY_CONFIGS["q_small"], seed=2, family="F2")
    st, ln = R.chunk_segments(np.array([3, 9, 17, 30]), qi.chunk_start, qi.chunk_len)
    a = _call(qi, st, ln)
    b = _call(qi, st[::-1], ln[::-1])
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=0, atol=1e-13)


def test_gather_attention_split_segments_merge_to_whole():
    """Attention over sink+segments+tail equals the LSE merge of the parts."""
    qi = make_query_inputs(QUERY_CONFIGS["q_small"], seed=3, family="F2")
    st, ln = R.chunk_segments(np.array([2, 5, 11]), qi.chunk_start, qi.chunk_len)
    whole = _call(qi, st, ln)
    # parts: the first segment, the other two segments (plain softmax attention
    # over their keys, fully visible), and sink + causal tail with no segment
    sh = qi.shape
    stk, stv = (f64(x) for x in qi.store_kv())
    g = sh.num_q_heads // sh.num_kv_heads
    outs, lses = [], []
    for part in (slice(0, 1), slice(1, 3)):
        slots = [p for a, n in zip(st[part], ln[part]) for p in range(int(a), int(a) + int(n))]
        o = np.zeros((sh.q_len, sh.num_q_heads, sh.head_dim))
        l = np.zeros((sh.num_q_heads, sh.q_len))
        for h in range(sh.num_q_heads):
            kv = h // g
            keys = stk[slots, kv]
            vals = stv[slots, kv]
            vis = np.ones((sh.q_len, len(slots)), dtype=bool)
            o[:, h], l[h] = oracle.softmax_attention(f64(qi.q)[:, h], keys, vals, vis, 1 / math.sqrt(sh.head_dim))
        outs.append(o)
        lses.append(l.T)
    # the rest: sink + tail only
    o3, l3 = R.gather_attention(f64(qi.q), f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k), f64(qi.sink_v),
                                stk, stv, [], [])
    outs.append(o3)
    lses.append(l3.T)
    mo, ml = oracle.lse_merge(outs, lses)
    np.testing.assert_allclose(mo, whole[0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(ml.T, whole[1], rtol=0, atol=1e-12)


def test_decode_row_equals_last_prefill_row():
    """A decode step (one query row, the newest tail token) equals the last row
    of the prefill over the same tail."""
    qi = make_query_inputs(QUERY_CONFIGS["q_gqa7"], seed=4, family="F2")
    st, ln = R.chunk_segments(np.array([0, 7, 8]), qi.chunk_start, qi.chunk_len)
    stk, stv = (f64(x) for x in qi.store_kv())
    q = f64(qi.q)
    full = R.gather_attention(q, f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k), f64(qi.sink_v), stk, stv, st, ln)
    one = R.gather_attention(q[-1:], f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k), f64(qi.sink_v), stk, stv, st, ln)
    np.testing.assert_allclose(one[0][0], full[0][-1], rtol=0, atol=1e-13)
    np.testing.assert_allclose(one[1][:, 0], full[1][:, -1], rtol=0, atol=1e-13)


def test_gather_over_the_window_equals_chunk_prefill():
    """Segments that list the visible window of a linear history, with the
    chunk as the tail and every chunk row a query row, reproduce the bounded
    chunk prefill (a separately pinned function)."""
    inp = make_chunk_inputs(CONFIGS["tiny"], seed=5, family="F2")
    a = to_f64(inp)
    sh = inp.shape
    wv = sh.visible_window
    n = a["hist_k"].shape[0]
    ref_o, ref_l = oracle.chunk_prefill_attention(**a)
    # the window as two segments of the stored history
    cut = wv // 3
    st = [n - wv, n - wv + cut]
    ln = [cut, wv - cut]
    out, lse = R.gather_attention(a["q"], a["k_chunk"], a["v_chunk"], a["sink_k"], a["sink_v"],
                                  a["hist_k"], a["hist_v"], st, ln)
    np.testing.assert_allclose(out, ref_o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, ref_l, rtol=0, atol=1e-12)


def test_single_visible_key_returns_its_value():
    qi = make_query_inputs(dataclasses.replace(QUERY_CONFIGS["q_tiny"], sink_len=0, q_len=1, tail_len=1), seed=6)
    stk, stv = (f64(x) for x in qi.store_kv())
    out, lse = R.gather_attention(f64(qi.q), f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k), f64(qi.sink_v),
                                  stk, stv, [], [])
    assert np.array_equal(out[0, 0], f64(qi.tail_v)[0, 0])
    z = f64(qi.q)[0, 0] @ f64(qi.tail_k)[0, 0] / math.sqrt(64)
    assert abs(lse[0, 0] - z) <= 1e-15


def test_rows_sum_to_one_and_constant_values():
    qi = make_query_inputs(QUERY_CONFIGS["q_small"], seed=7, family="F2")
    st, ln = R.chunk_segments(np.array([1, 2, 3]), qi.chunk_start, qi.chunk_len)
    stk, _ = (f64(x) for x in qi.store_kv())
    ones = lambda x: np.full(x.shape, 2.5)
    out, _ = R.gather_attention(f64(qi.q), f64(qi.tail_k), ones(qi.tail_v), f64(qi.sink_k), ones(qi.sink_v),
                                stk, ones(stk), st, ln)
    np.testing.assert_allclose(out, 2.5, rtol=0, atol=1e-13)


def test_zero_query_lse_counts_visible_keys():
    qi = make_query_inputs(QUERY_CONFIGS["q_small"], seed=8)
    st, ln = R.chunk_segments(np.array([0, 4]), qi.chunk_start, qi.chunk_len)
    stk, stv = (f64(x) for x in qi.store_kv())
    sh = qi.shape
    _, lse = R.gather_attention(np.zeros(f64(qi.q).shape), f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k),
                                f64(qi.sink_v), stk, stv, st, ln)
    n_vis = sh.sink_len + int(np.sum(ln)) + sh.tail_len - sh.q_len + 1 + np.arange(sh.q_len)
    np.testing.assert_allclose(lse, np.tile(np.log(n_vis), (sh.num_q_heads, 1)), rtol=0, atol=1e-13)


def test_segment_outside_the_store_is_an_error():
    qi = make_query_inputs(QUERY_CONFIGS["q_tiny"], seed=0)
    stk, stv = (f64(x) for x in qi.store_kv())
    with pytest.raises(ValueError):
        R.gather_attention(f64(qi.q), f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k), f64(qi.sink_v),
                           stk, stv, [qi.store_len - 2], [3])
