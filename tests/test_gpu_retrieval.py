"""GPU parity of query-side retrieval and the gathered short-query attention
against the oracle (paper, Sec. 3, query-time decoding; query rows of
Eq. (4)).

Bounds used here, derived from the arithmetic:
  * token mean: fp32 sums of at most L terms in a fixed order, then one
    division: |err| <= (L + 2) * 2^-24 * mean|x| + 2^-24 |mean| per column.
  * cosine: fp32 dot product and norms of dm terms; by Cauchy-Schwarz each
    sum's rounding error is at most dm * 2^-24 of |q||c|, so
    |err| <= (3 dm + 8) * 2^-24.
  * top-k: an integer decision taken on floating-point scores.  On the GPU's
    own fp32 scores the oracle's rule (same precision) must give exactly the
    GPU's selection.  Against the fp64 scores, the selection must equal the
    oracle's wherever the k-th and (k+1)-th scores are further apart than
    twice the cosine bound, and otherwise stay within that bound of it.
  * gathered attention: the derived per-element bounds of tests/_bounds.py
    (bf16 probabilities, fp32 logits and sums, the log-sum-exp merge of the
    key-range parts), output and LSE, as for the chunk prefill.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_19849_amd as vico
from synth import CONFIGS, QUERY_CONFIGS, QueryShape, make_chunk_inputs, make_query_inputs, make_tokens
from tests._bounds import Bound, chunk_bound, gather_bound
from tests._gpu import check_bf16, check_f1, check_f32, dev
from tests._util import ring_from_inputs, to_f64

pytestmark = pytest.mark.gpu

f64 = oracle.bf16_bits_to_f64
U = 2.0 ** -24


# ---------------------------------------------------------------- token mean

@pytest.mark.parametrize("L,dm", [(1, 8), (37, 264), (5, 2048), (1024, 3584), (3000, 512)])
def test_token_mean(L, dm):
    x = make_tokens(L, dm, seed=L, offset=0.5)
    out = torch.empty(dm, dtype=torch.float32, device="cuda")
    vico.vico_token_mean(dev(x), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    xf = f64(x)
    ref = oracle.token_mean(xf)
    bound = (L + 2) * U * np.mean(np.abs(xf), axis=0) + U * np.abs(ref)
    assert np.all(np.abs(got - ref) <= bound)


def test_token_mean_of_identical_rows_is_exact():
    row = make_tokens(1, 1024, seed=9)
    x = np.repeat(row, 64, axis=0)          # 64 * v is exact in fp32 for bf16 v, and so is the division
    out = torch.empty(1024, dtype=torch.float32, device="cuda")
    vico.vico_token_mean(dev(x), out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().astype(np.float64), f64(row)[0])


# ---------------------------------------------------------------- cosine scores

def _scores_gpu(qf, cf):
    s = torch.empty(cf.shape[0], dtype=torch.float32, device="cuda")
    vico.vico_chunk_scores(torch.from_numpy(qf).cuda(), torch.from_numpy(cf).cuda(), s)
    torch.cuda.synchronize()
    return s.cpu().numpy()


@pytest.mark.parametrize("name", ["q_small", "q_7b"])
def test_chunk_scores(name):
    qi = make_query_inputs(QUERY_CONFIGS[name], seed=2)
    dm = qi.shape.feat_dim
    qf = (qi.chunk_feat[3] + np.random.default_rng(5).standard_normal(dm).astype(np.float32)).astype(np.float32)
    got = _scores_gpu(qf, qi.chunk_feat).astype(np.float64)
    ref = oracle.cosine_scores(qf.astype(np.float64), qi.chunk_feat.astype(np.float64))
    assert np.max(np.abs(got - ref)) <= (3 * dm + 8) * U


def test_chunk_scores_special_rows():
    dm = 64
    rng = np.random.default_rng(0)
    q = rng.standard_normal(dm).astype(np.float32)
    cf = np.stack([q * 3, -q, np.zeros(dm, np.float32), rng.standard_normal(dm).astype(np.float32)])
    got = _scores_gpu(q, cf)
    tol = (3 * dm + 8) * U
    assert abs(got[0] - 1) <= tol and abs(got[1] + 1) <= tol
    assert got[2] == 0 and not np.signbit(got[2])
    assert np.all(_scores_gpu(np.zeros(dm, np.float32), cf) == 0)


# ---------------------------------------------------------------- top-k

def _topk_gpu(scores, k, tau=-math.inf, chunk_start=None, chunk_len=None):
    N = len(scores)
    sc = torch.from_numpy(np.asarray(scores, dtype=np.float32)).cuda()
    oc = torch.full((k,), 12345, dtype=torch.int32, device="cuda")
    os_ = torch.zeros(k, dtype=torch.float32, device="cuda")
    cnt = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    kw = {}
    if chunk_start is not None:
        kw = dict(chunk_start=torch.from_numpy(np.asarray(chunk_start, np.int64)).cuda(),
                  chunk_len=torch.from_numpy(np.asarray(chunk_len, np.int32)).cuda(),
                  seg_start=torch.full((k,), -1, dtype=torch.int64, device="cuda"),
                  seg_len=torch.full((k,), -1, dtype=torch.int32, device="cuda"))
    vico.vico_topk_chunks(sc, k, oc, os_, cnt, min_score=tau, **kw)
    torch.cuda.synchronize()
    n = int(cnt.item())
    res = dict(count=n, chunks=oc.cpu().numpy(), scores=os_.cpu().numpy())
    if kw:
        res["seg_start"] = kw["seg_start"].cpu().numpy()
        res["seg_len"] = kw["seg_len"].cpu().numpy()
    return res


def _check_topk_exact(scores32, k, tau=-math.inf, table=True):
    N = len(scores32)
    rng = np.random.default_rng(N + k)
    lens = rng.integers(1, 900, N)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    r = _topk_gpu(scores32, k, tau, starts if table else None, lens if table else None)
    want = oracle.select_chunks(np.asarray(scores32, np.float64), k, tau)
    n = len(want)
    assert r["count"] == n
    assert np.array_equal(r["chunks"][:n], want)
    assert np.all(r["chunks"][n:] == -1)
    assert np.array_equal(r["scores"][:n].view(np.uint32), np.asarray(scores32, np.float32)[want].view(np.uint32)) \
        or np.array_equal(r["scores"][:n], np.asarray(scores32, np.float32)[want])
    assert np.all(np.isneginf(r["scores"][n:]))
    if table:
        assert np.array_equal(r["seg_start"][:n], starts[want]) and np.array_equal(r["seg_len"][:n], lens[want])
        assert np.all(r["seg_len"][n:] == 0) and np.all(r["seg_start"][n:] == 0)


@pytest.mark.parametrize("N", [1, 5, 256, 257, 1000, 1024, 5000, 100000])   # 256 threads up to 256 scores
@pytest.mark.parametrize("k", [1, 7, 32, 2048])
def test_topk_matches_oracle_rule_on_fp32_scores(N, k):
    rng = np.random.default_rng(N * 7 + k)
    s = rng.uniform(-1, 1, N).astype(np.float32)
    s[: N // 3] = np.round(s[: N // 3], 2)          # many exact ties
    _check_topk_exact(s, k)


@pytest.mark.parametrize("tau", [0.3, 0.999, 2.0, -0.5])
def test_topk_threshold(tau):
    s = np.round(np.random.default_rng(3).uniform(-1, 1, 3000), 3).astype(np.float32)
    _check_topk_exact(s, 64, tau)


def test_topk_special_values():
    s = np.array([0.0, -0.0, np.nan, 0.5, -np.inf, np.inf, 0.5, -0.0, np.nan, 1e-30], dtype=np.float32)
    for k in (1, 2, 3, 4, 6, 8, 10):
        _check_topk_exact(s, k)
    _check_topk_exact(s, 3, table=False)


def test_topk_no_chunks():
    r = _topk_gpu(np.zeros(0, np.float32), 4)
    assert r["count"] == 0 and np.all(r["chunks"] == -1)


# ---------------------------------------------------------------- gathered attention

class DeviceQuery:
    def __init__(self, qi):
        self.qi = qi
        self.q, self.tk, self.tv = dev(qi.q), dev(qi.tail_k), dev(qi.tail_v)
        sh = qi.shape
        self.sk = dev(qi.sink_k) if sh.sink_len else None
        self.sv = dev(qi.sink_v) if sh.sink_len else None
        k, v = qi.store_kv()
        self.store_np = (k, v)
        self.gk, self.gv = dev(k), dev(v)

    def attend(self, seg_start, seg_len, out_dtype=torch.float32, num_splits=0, q_rows=None, hint=None):
        sh = self.qi.shape
        q = self.q if q_rows is None else self.q[-q_rows:].contiguous()
        Lq = q.shape[0]
        ss = torch.from_numpy(np.asarray(seg_start, np.int64)).cuda() if len(seg_start) else None
        sl = torch.from_numpy(np.asarray(seg_len, np.int32)).cuda() if len(seg_len) else None
        if hint is None:
            hint = int(np.sum(np.maximum(np.asarray(seg_len, np.int64), 0))) if len(seg_len) else 0
        parts, wb = vico.vico_gather_plan(Lq, sh.tail_len, sh.sink_len, self.gk.shape[0], len(seg_start), hint,
                                          sh.num_q_heads, sh.num_kv_heads, sh.head_dim, num_splits)
        ws = torch.empty(max(wb, 1), dtype=torch.uint8, device="cuda") if wb else None
        out = torch.empty((Lq, sh.num_q_heads, sh.head_dim), dtype=out_dtype, device="cuda")
        lse = torch.empty((sh.num_q_heads, Lq), dtype=torch.float32, device="cuda")
        vico.vico_gather_attn(q, self.tk, self.tv, self.sk, self.sv, self.gk, self.gv, ss, sl, out, lse=lse,
                              workspace=ws, keys_hint=hint, num_splits=num_splits)
        torch.cuda.synchronize()
        return out.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64), parts

    def reference(self, seg_start, seg_len, q_rows=None, heads=None, scale=None, parts=1, sigma=False):
        """Oracle output, LSE and the derived bound; the oracle sees only the
        store rows the segments name (a compacted copy, same order)."""
        qi = self.qi
        q = f64(qi.q) if q_rows is None else f64(qi.q)[-q_rows:]
        k, v = self.store_np
        seg_start = np.asarray(seg_start, np.int64)
        seg_len = np.asarray(seg_len, np.int64)
        d = qi.shape.head_dim
        Hkv = qi.shape.num_kv_heads
        ck = f64(np.concatenate([k[a:a + n] for a, n in zip(seg_start, seg_len)] or [k[:0]]))
        cv = f64(np.concatenate([v[a:a + n] for a, n in zip(seg_start, seg_len)] or [v[:0]]))
        cs = np.concatenate([[0], np.cumsum(seg_len)[:-1]]).astype(np.int64) if len(seg_len) else seg_start
        args = (q, f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k).reshape(-1, Hkv, d),
                f64(qi.sink_v).reshape(-1, Hkv, d), ck.reshape(-1, Hkv, d), cv.reshape(-1, Hkv, d), cs, seg_len)
        ro, rl = oracle.gather_attention(*args, heads=heads, scale=scale)
        b = gather_bound(*args, heads=heads, scale=scale, parts=parts, sigma=sigma)
        return ro, rl, b


SMALL_Q = ["q_tiny", "q_small", "q_gqa7"]


@pytest.mark.parametrize("name", SMALL_Q)
@pytest.mark.parametrize("splits", [0, 1, 3, 7])
def test_gather_attention_parity(name, splits):
    qi = make_query_inputs(QUERY_CONFIGS[name], seed=11, family="F2")
    sel = oracle.select_chunks(np.random.default_rng(1).uniform(size=qi.shape.num_chunks), qi.shape.top_k)
    st, ln = oracle.chunk_segments(sel, qi.chunk_start, qi.chunk_len)
    d = DeviceQuery(qi)
    o, l, parts = d.attend(st, ln, num_splits=splits)
    ro, rl, b = d.reference(st, ln, parts=parts)
    check_f32(o, ro, b, l, rl)
    if splits:
        assert parts == splits


@pytest.mark.parametrize("name", SMALL_Q)
def test_gather_attention_bf16_out(name):
    qi = make_query_inputs(QUERY_CONFIGS[name], seed=12, family="F2")
    sel = oracle.select_chunks(np.random.default_rng(2).uniform(size=qi.shape.num_chunks), qi.shape.top_k)
    st, ln = oracle.chunk_segments(sel, qi.chunk_start, qi.chunk_len)
    d = DeviceQuery(qi)
    o, _, parts = d.attend(st, ln, out_dtype=torch.bfloat16)
    ro, _, b = d.reference(st, ln, parts=parts)
    check_bf16(o, ro, b)


@pytest.mark.parametrize("splits", [0, 4])
def test_decode_step(splits):
    """One query row (the newest tail token), as in token-by-token decoding."""
    qi = make_query_inputs(QUERY_CONFIGS["q_gqa7"], seed=13, family="F2")
    st, ln = oracle.chunk_segments(np.array([0, 5, 6, 20]), qi.chunk_start, qi.chunk_len)
    d = DeviceQuery(qi)
    o, l, parts = d.attend(st, ln, q_rows=1, num_splits=splits)
    ro, rl, b = d.reference(st, ln, q_rows=1, parts=parts)
    check_f32(o, ro, b, l, rl)


def test_decode_step_replays_as_a_graph():
    """A decode step captured into a HIP graph (the library launches kernels
    only: no memset, copy or allocation) replays the eager result exactly,
    replay after replay, with other eager work of the same buffers between."""
    qi = make_query_inputs(QUERY_CONFIGS["q_gqa7"], seed=15, family="F2")
    sh = qi.shape
    d = DeviceQuery(qi)
    q = d.q[-1:].contiguous()
    tables = [oracle.chunk_segments(np.array(c), qi.chunk_start, qi.chunk_len) for c in ([0, 5, 6, 20], [1, 2, 9])]
    segs = [(torch.from_numpy(st.astype(np.int64)).cuda(), torch.from_numpy(ln.astype(np.int32)).cuda())
            for st, ln in tables]
    hint = max(int(ln.sum()) for _, ln in tables)
    parts, wb = vico.vico_gather_plan(1, sh.tail_len, sh.sink_len, d.gk.shape[0], 4, hint, sh.num_q_heads,
                                      sh.num_kv_heads, sh.head_dim)
    assert parts > 1                  # the merge kernel is part of the graph
    ws = torch.empty(wb, dtype=torch.uint8, device="cuda")
    out = torch.empty((1, sh.num_q_heads, sh.head_dim), dtype=torch.float32, device="cuda")
    lse = torch.empty((sh.num_q_heads, 1), dtype=torch.float32, device="cuda")

    def step(i):
        vico.vico_gather_attn(q, d.tk, d.tv, d.sk, d.sv, d.gk, d.gv, segs[i][0], segs[i][1], out, lse=lse,
                              workspace=ws, keys_hint=hint)

    eager = []
    for i in range(2):
        step(i)
        torch.cuda.synchronize()
        eager.append((out.clone(), lse.clone()))
    ro, rl, b = d.reference(*tables[0], q_rows=1, parts=parts)
    check_f32(eager[0][0].cpu().numpy().astype(np.float64), ro, b, eager[0][1].cpu().numpy().astype(np.float64), rl)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        step(0)                       # warm-up on the capture stream
        torch.cuda.current_stream().synchronize()
        with torch.cuda.graph(graph, stream=side):
            step(0)
    torch.cuda.synchronize()
    for _ in range(3):
        step(1)                       # eager call of another table, same buffers
        torch.cuda.synchronize()
        assert torch.equal(out, eager[1][0]) and torch.equal(lse, eager[1][1])
        out.zero_()
        lse.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager[0][0]) and torch.equal(lse, eager[0][1])


@pytest.mark.parametrize("scale", [0.03, 0.5])
def test_gather_explicit_softmax_scale(scale):
    """softmax_scale > 0 replaces 1/sqrt(d) on the gathered path too (4 query
    rows, F2 inputs), fp32 output and LSE against the oracle at that scale."""
    qi = make_query_inputs(QUERY_CONFIGS["q_gqa7"], seed=16, family="F2")
    sh = qi.shape
    st, ln = oracle.chunk_segments(np.array([1, 4, 7]), qi.chunk_start, qi.chunk_len)
    d = DeviceQuery(qi)
    Lq = 4
    q = d.q[-Lq:].contiguous()
    hint = int(ln.sum())
    parts, wb = vico.vico_gather_plan(Lq, sh.tail_len, sh.sink_len, d.gk.shape[0], len(st), hint, sh.num_q_heads,
                                      sh.num_kv_heads, sh.head_dim)
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
    out = torch.empty((Lq, sh.num_q_heads, sh.head_dim), dtype=torch.float32, device="cuda")
    lse = torch.empty((sh.num_q_heads, Lq), dtype=torch.float32, device="cuda")
    vico.vico_gather_attn(q, d.tk, d.tv, d.sk, d.sv, d.gk, d.gv, torch.from_numpy(st.astype(np.int64)).cuda(),
                          torch.from_numpy(ln.astype(np.int32)).cuda(), out, lse=lse, workspace=ws,
                          keys_hint=hint, softmax_scale=scale)
    torch.cuda.synchronize()
    ro, rl, b = d.reference(st, ln, q_rows=Lq, scale=scale, parts=parts)
    check_f32(out.cpu().numpy().astype(np.float64), ro, b, lse.cpu().numpy().astype(np.float64), rl)


def test_no_segments_attends_sink_and_tail():
    qi = make_query_inputs(QUERY_CONFIGS["q_small"], seed=14, family="F2")
    d = DeviceQuery(qi)
    o, l, parts = d.attend([], [])
    ro, rl, b = d.reference([], [], parts=parts)
    check_f32(o, ro, b, l, rl)


def test_segments_are_clipped_to_the_store():
    """Zero-length, negative, overlapping and out-of-store segments: the kernel
    attends to the parts inside the store, exactly as the clipped table."""
    qi = make_query_inputs(QUERY_CONFIGS["q_small"], seed=15, family="F2")
    n = qi.store_len
    st = np.array([5, 100, n - 10, -30, 40, 2 * n, 300, 300], np.int64)
    ln = np.array([0, 50, 25, 40, -3, 10, 64, 64], np.int64)
    lo = np.clip(st, 0, n)
    hi = np.clip(st + ln, 0, n)
    keep = hi > lo
    d = DeviceQuery(qi)
    o, l, parts = d.attend(st, ln)
    ro, rl, b = d.reference(lo[keep], (hi - lo)[keep], parts=parts)
    check_f32(o, ro, b, l, rl)


def test_many_tiny_segments():
    """Single-token segments in scattered order: every key row of a tile comes
    from a different place."""
    qi = make_query_inputs(QUERY_CONFIGS["q_small"], seed=16, family="F2")
    rng = np.random.default_rng(4)
    st = rng.permutation(qi.store_len)[:1500].astype(np.int64)
    ln = rng.integers(0, 3, 1500).astype(np.int64)
    lo, hi = np.clip(st, 0, qi.store_len), np.clip(st + ln, 0, qi.store_len)
    d = DeviceQuery(qi)
    o, l, parts = d.attend(st, ln, num_splits=5)
    ro, rl, b = d.reference(lo, np.maximum(hi - lo, 0), parts=parts)
    check_f32(o, ro, b, l, rl)


def test_d64_and_mha():
    sh = QueryShape(4, 4, 64, 3, 128, 20, 10, 150, 5, 8, 6)
    qi = make_query_inputs(sh, seed=17, family="F2")
    sel = oracle.select_chunks(np.random.default_rng(5).uniform(size=sh.num_chunks), sh.top_k)
    st, ln = oracle.chunk_segments(sel, qi.chunk_start, qi.chunk_len)
    d = DeviceQuery(qi)
    o, l, parts = d.attend(st, ln, num_splits=2)
    ro, rl, b = d.reference(st, ln, parts=parts)
    check_f32(o, ro, b, l, rl)


def test_long_query_spans_two_row_tiles():
    """g * Lq > 256 packed rows: two row tiles per KV head."""
    sh = QueryShape(14, 2, 128, 16, 256, 30, 40, 300, 50, 60, 8)
    qi = make_query_inputs(sh, seed=18, family="F2")
    sel = oracle.select_chunks(np.random.default_rng(6).uniform(size=sh.num_chunks), sh.top_k)
    st, ln = oracle.chunk_segments(sel, qi.chunk_start, qi.chunk_len)
    d = DeviceQuery(qi)
    for splits in (0, 3):
        o, l, parts = d.attend(st, ln, num_splits=splits)
        ro, rl, b = d.reference(st, ln, parts=parts)
        check_f32(o, ro, b, l, rl)


def test_gather_over_ring_window_equals_chunk_prefill():
    """The bounded window of a ring, given as its (up to) two slot ranges, with
    the chunk as the tail: the same result as the chunk prefill oracle."""
    inp = make_chunk_inputs(CONFIGS["tiny"], seed=19, family="F2")
    sh = inp.shape
    rk, rv = ring_from_inputs(inp)
    wv = sh.visible_window
    ws = (sh.hist_len - wv) % sh.ring_slots
    first = min(wv, sh.ring_slots - ws)
    st, ln = [ws, 0], [first, wv - first]
    q, tk, tv = dev(inp.q), dev(inp.k_chunk), dev(inp.v_chunk)
    out = torch.empty((sh.chunk_len, sh.num_q_heads, sh.head_dim), dtype=torch.float32, device="cuda")
    lse = torch.empty((sh.num_q_heads, sh.chunk_len), dtype=torch.float32, device="cuda")
    vico.vico_gather_attn(q, tk, tv, dev(inp.sink_k), dev(inp.sink_v), dev(rk), dev(rv),
                          torch.tensor(st, dtype=torch.int64, device="cuda"),
                          torch.tensor(ln, dtype=torch.int32, device="cuda"), out, lse=lse, keys_hint=wv)
    torch.cuda.synchronize()
    parts = vico.vico_gather_plan(sh.chunk_len, sh.chunk_len, sh.sink_len, sh.ring_slots, 2, wv, sh.num_q_heads,
                                  sh.num_kv_heads, sh.head_dim)[0]
    x = to_f64(inp)
    ro, rl = oracle.chunk_prefill_attention(**x)
    check_f32(out.cpu().numpy().astype(np.float64), ro, chunk_bound(x, parts=parts),
              lse.cpu().numpy().astype(np.float64), rl)


# ---------------------------------------------------------------- whole query path at full size

@pytest.mark.parametrize("name", ["q_7b", "q_3b"])
def test_query_path_full_size(name):
    """Query mean -> scores over all stored chunks -> top-k with its segment
    table -> gathered attention, all on the device with no host round trip;
    checked stage by stage against the oracle."""
    qi = make_query_inputs(QUERY_CONFIGS[name], seed=0, family="F2")
    sh = qi.shape
    d = DeviceQuery(qi)
    qx = dev(qi.query_x)
    qf = torch.empty(sh.feat_dim, dtype=torch.float32, device="cuda")
    feats = torch.from_numpy(qi.chunk_feat).cuda()
    scores = torch.empty(sh.num_chunks, dtype=torch.float32, device="cuda")
    oc = torch.empty(sh.top_k, dtype=torch.int32, device="cuda")
    os_ = torch.empty(sh.top_k, dtype=torch.float32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    ss = torch.empty(sh.top_k, dtype=torch.int64, device="cuda")
    sl = torch.empty(sh.top_k, dtype=torch.int32, device="cuda")
    vico.vico_token_mean(qx, qf)
    vico.vico_chunk_scores(qf, feats, scores)
    vico.vico_topk_chunks(scores, sh.top_k, oc, os_, cnt, chunk_start=torch.from_numpy(qi.chunk_start).cuda(),
                          chunk_len=torch.from_numpy(qi.chunk_len.astype(np.int32)).cuda(), seg_start=ss,
                          seg_len=sl)
    hint = sh.top_k * (sh.chunk_lo + sh.chunk_hi) // 2
    parts, wb = vico.vico_gather_plan(sh.q_len, sh.tail_len, sh.sink_len, qi.store_len, sh.top_k, hint,
                                      sh.num_q_heads, sh.num_kv_heads, sh.head_dim)
    ws = torch.empty(max(wb, 1), dtype=torch.uint8, device="cuda")
    out = torch.empty((sh.q_len, sh.num_q_heads, sh.head_dim), dtype=torch.float32, device="cuda")
    lse = torch.empty((sh.num_q_heads, sh.q_len), dtype=torch.float32, device="cuda")
    vico.vico_gather_attn(d.q, d.tk, d.tv, d.sk, d.sv, d.gk, d.gv, ss, sl, out, lse=lse, workspace=ws,
                          keys_hint=hint)
    torch.cuda.synchronize()

    # stage 1-2: scores within the cosine bound of the fp64 pipeline
    ref_qf = oracle.token_mean(f64(qi.query_x))
    ref_s = oracle.cosine_scores(ref_qf, qi.chunk_feat.astype(np.float64))
    got_s = scores.cpu().numpy().astype(np.float64)
    tol = (3 * sh.feat_dim + 8) * U + 1e-6            # + the query mean's own rounding
    assert np.max(np.abs(got_s - ref_s)) <= tol
    # stage 3: exact on the kernel's scores; valid against the fp64 scores
    sel = oc.cpu().numpy()[: int(cnt.item())]
    assert np.array_equal(sel, oracle.select_chunks(scores.cpu().numpy().astype(np.float64), sh.top_k))
    order = np.sort(ref_s)[::-1]
    kth = order[sh.top_k - 1]
    assert np.all(ref_s[sel] >= kth - 2 * tol)
    out_set = np.setdiff1d(np.arange(sh.num_chunks), sel)
    assert np.all(ref_s[out_set] <= kth + 2 * tol)
    if order[sh.top_k - 1] - order[sh.top_k] > 2 * tol:
        assert np.array_equal(sel, oracle.select_chunks(ref_s, sh.top_k))
    st, ln = oracle.chunk_segments(sel, qi.chunk_start, qi.chunk_len)
    assert np.array_equal(ss.cpu().numpy(), st) and np.array_equal(sl.cpu().numpy(), ln)
    # stage 4: attention over the selected chunks, every row and head
    ro, rl, b = d.reference(st, ln, parts=parts)
    check_f32(out.cpu().numpy().astype(np.float64), ro, b, lse.cpu().numpy().astype(np.float64), rl)


def test_store_at_the_32bit_offset_limit():
    """Largest store the gathered attention addresses (2^31 bytes per K/V
    tensor less one row: 8388607 slots of one d128 head).  All keys are zero,
    so each query row's output is the plain mean of the V rows it sees (sink,
    segments, causal tail) and its LSE is ln(count).  Store V rows carry a
    slot-hashed 0/1 pattern and the segments include the store's last slots,
    so a misaddressed or out-of-range read changes the mean."""
    Hq, Hkv, D, S, T, Lq = 7, 1, 128, 16, 64, 2
    cap = (1 << 31) // (Hkv * D * 2) - 1
    dev = "cuda"
    g = torch.Generator().manual_seed(9)
    marks = lambda x: ((x * 2654435761) >> 13) & 1
    cvec = ((torch.arange(D) % 7 - 3) / 4).to(torch.bfloat16)
    gk = torch.zeros((cap, Hkv, D), dtype=torch.bfloat16, device=dev)
    gv = (marks(torch.arange(cap, device=dev)).to(torch.bfloat16)[:, None] * cvec.to(dev)[None, :]).reshape(cap, Hkv, D)
    sk = torch.zeros((S, Hkv, D), dtype=torch.bfloat16, device=dev)
    sv = torch.randn((S, Hkv, D), generator=g).to(torch.bfloat16)
    tk = torch.zeros((T, Hkv, D), dtype=torch.bfloat16, device=dev)
    tv = torch.randn((T, Hkv, D), generator=g).to(torch.bfloat16)
    q = torch.randn((Lq, Hq, D), generator=g).to(torch.bfloat16).to(dev)
    st = np.array([cap - 5000, 0, 4_000_000], np.int64)
    ln = np.array([5000, 3000, 2000], np.int32)
    hint = int(ln.sum())
    parts, wb = vico.vico_gather_plan(Lq, T, S, cap, len(st), hint, Hq, Hkv, D)
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device=dev)
    out = torch.empty((Lq, Hq, D), dtype=torch.float32, device=dev)
    lse = torch.empty((Hq, Lq), dtype=torch.float32, device=dev)
    vico.vico_gather_attn(q, tk, tv.to(dev), sk, sv.to(dev), gk, gv, torch.from_numpy(st).to(dev),
                          torch.from_numpy(ln).to(dev), out, lse=lse, workspace=ws, keys_hint=hint)
    torch.cuda.synchronize()
    slots = np.concatenate([np.arange(a, a + n, dtype=np.int64) for a, n in zip(st, ln)])
    seg_sum = float(marks(slots).sum()) * cvec.double().numpy()
    sv64, tv64 = sv.double().numpy()[:, 0], tv.double().numpy()[:, 0]
    o = out.cpu().double().numpy()
    l = lse.cpu().double().numpy()
    seg_abs = float(marks(slots).sum()) * cvec.double().abs().numpy()
    for i in range(Lq):
        vis_tail = T - Lq + i + 1
        n = S + hint + vis_tail
        mean = (sv64.sum(0) + seg_sum + tv64[:vis_tail].sum(0)) / n
        # every logit is exactly 0, so every probability is exactly 1: only
        # the fp32 sums and the merge round (the derived bound with no logit error)
        A = (np.abs(sv64).sum(0) + seg_abs + np.abs(tv64[:vis_tail]).sum(0)) / n
        b = Bound(A[None, None, :], np.zeros((1, 1)), np.zeros((1, 1)), n, parts)
        assert np.all(np.abs(o[i] - mean[None, :]) <= b.f32(mean[None, None, :])[0])
        assert np.all(np.abs(l[:, i] - np.log(n)) <= b.lse(np.log(n)))


@pytest.mark.parametrize("family,query_seed", [("F1", 0), ("F1", 5), ("F2", 0)])
def test_decode_step_full_size(family, query_seed):
    """One decode step at full size, as timed: 7B heads (28 query, 4 KV,
    d 128), a query row over sink 64 + the 32 chunks retrieved from a
    256-chunk store (336 MB of K/V) + a 64-token tail, with the key-range
    split the planner picks for it; retrieval on the device, bf16 output.
    Every head's output element and LSE against the derived bound (for the
    N(0,1)/sqrt(d) family also the statistical one)."""
    base = dataclasses.replace(QUERY_CONFIGS["q_7b"], tail_len=64)
    qi = make_query_inputs(base, seed=0, family=family, query_seed=query_seed)
    sh = qi.shape
    d = DeviceQuery(qi)
    qf = torch.empty(sh.feat_dim, dtype=torch.float32, device="cuda")
    scores = torch.empty(sh.num_chunks, dtype=torch.float32, device="cuda")
    oc = torch.empty(sh.top_k, dtype=torch.int32, device="cuda")
    os_ = torch.empty(sh.top_k, dtype=torch.float32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    ss = torch.empty(sh.top_k, dtype=torch.int64, device="cuda")
    sl = torch.empty(sh.top_k, dtype=torch.int32, device="cuda")
    vico.vico_token_mean(dev(qi.query_x), qf)
    vico.vico_chunk_scores(qf, torch.from_numpy(qi.chunk_feat).cuda(), scores)
    vico.vico_topk_chunks(scores, sh.top_k, oc, os_, cnt, chunk_start=torch.from_numpy(qi.chunk_start).cuda(),
                          chunk_len=torch.from_numpy(qi.chunk_len.astype(np.int32)).cuda(), seg_start=ss,
                          seg_len=sl)
    hint = sh.top_k * (sh.chunk_lo + sh.chunk_hi) // 2
    parts, wb = vico.vico_gather_plan(1, sh.tail_len, sh.sink_len, qi.store_len, sh.top_k, hint,
                                      sh.num_q_heads, sh.num_kv_heads, sh.head_dim)
    assert parts > 1                  # the split and the merge are part of the step
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
    out = torch.empty((1, sh.num_q_heads, sh.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((sh.num_q_heads, 1), dtype=torch.float32, device="cuda")
    vico.vico_gather_attn(d.q[-1:].contiguous(), d.tk, d.tv, d.sk, d.sv, d.gk, d.gv, ss, sl, out, lse=lse,
                          workspace=ws, keys_hint=hint)
    torch.cuda.synchronize()
    n = int(cnt.item())
    assert n == sh.top_k
    st, ln = ss.cpu().numpy(), sl.cpu().numpy().astype(np.int64)
    sel = oc.cpu().numpy()[:n]
    assert np.array_equal(st, qi.chunk_start[sel]) and np.array_equal(ln, qi.chunk_len[sel])
    o = out.float().cpu().numpy().astype(np.float64)
    l = lse.cpu().numpy().astype(np.float64)
    ro, rl, b = d.reference(st, ln, q_rows=1, parts=parts, sigma=family == "F1")
    if family == "F1":
        check_f1(o, ro, b, out_bf16=True)
    else:
        check_bf16(o, ro, b)
    assert np.all(np.abs(l - rl) <= b.lse(rl))
