"""The fixtures of tests/golden/ (written by tests/golden/make_golden.py from
the oracle) against closed forms computed here without the oracle, and
against the oracle as it stands (a change to its arithmetic shows up here
first).  CPU only."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import paper_2606_19849_amd as vico

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def visible_bases(case, i):
    """Base values of the keys chunk row i sees, listed key by key: the sink,
    the newest min(W, H) history positions (all of them for W < 0), chunk
    tokens 0..i."""
    S, H, W = case["sink_len"], case["hist_len"], case["window"]
    first = 0 if W < 0 else max(0, H - W)
    return [100 + s for s in range(S)] + [10 + p for p in range(first, H)] + [60 + j for j in range(i + 1)]


@pytest.mark.parametrize("case", load("attention_uniform.json")["cases"], ids=lambda c: c["name"])
def test_attention_uniform_fixture(case):
    Hq = case["num_q_heads"]
    for i in range(case["chunk_len"]):
        keys = visible_bases(case, i)
        want = Fraction(sum(keys), len(keys))
        for h in range(Hq):
            assert case["out_column0"][i][h] == pytest.approx(float(want), rel=0, abs=1e-12)
            assert case["lse"][h][i] == pytest.approx(math.log(len(keys)), rel=0, abs=1e-12)
    # the oracle as it stands
    Hkv, d, S, H, W, C = (case[k] for k in ("num_kv_heads", "head_dim", "sink_len", "hist_len", "window", "chunk_len"))
    rows = lambda base, n: np.stack([np.full((Hkv, d), base + i) + np.arange(d) for i in range(n)]) \
        if n else np.zeros((0, Hkv, d))
    z = lambda n: np.zeros((n, Hkv, d))
    out, lse = oracle.chunk_prefill_attention(np.zeros((C, Hq, d)), z(C), rows(60, C), z(S), rows(100, S), z(H),
                                              rows(10, H), H, W)
    assert np.allclose(out[:, :, 0], case["out_column0"], rtol=0, atol=1e-12)
    assert np.allclose(out - out[:, :, :1], np.arange(d), rtol=0, atol=1e-9)     # column c = column 0 + c
    assert np.allclose(lse, case["lse"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("case", load("gather_uniform.json")["cases"], ids=lambda c: c["name"])
def test_gather_uniform_fixture(case):
    S, T, Lq, Hq = case["sink_len"], case["tail_len"], case["q_len"], case["num_q_heads"]
    b = case["bases"]
    cap = case["store_slots"]
    store_keys = [b["store"] + slot for a, n in zip(case["table_start"], case["table_len"])
                  for slot in range(a, a + n) if 0 <= slot < cap]         # the part of each entry inside the store
    for i in range(Lq):
        keys = [b["sink"] + s for s in range(S)] + store_keys + [b["tail"] + t for t in range(T - Lq + i + 1)]
        want = Fraction(sum(keys), len(keys))
        for h in range(Hq):
            assert case["out_column0"][i][h] == pytest.approx(float(want), rel=0, abs=1e-12)
            assert case["lse"][h][i] == pytest.approx(math.log(len(keys)), rel=0, abs=1e-12)
    Hkv, d = case["num_kv_heads"], case["head_dim"]
    rows = lambda base, n: np.stack([np.full((Hkv, d), base + i) + np.arange(d) for i in range(n)])
    z = lambda n: np.zeros((n, Hkv, d))
    out, lse = oracle.gather_attention(np.zeros((Lq, Hq, d)), z(T), rows(b["tail"], T), z(S), rows(b["sink"], S),
                                       z(cap), rows(b["store"], cap), case["seg_start"], case["seg_len"])
    assert np.allclose(out[:, :, 0], case["out_column0"], rtol=0, atol=1e-12)
    assert np.allclose(lse, case["lse"], rtol=0, atol=1e-12)


def test_acn_window_fixture():
    g = load("acn_windows.json")
    starts = g["chunk_starts"]
    lens = [b - a for a, b in zip(starts, starts[1:])]
    for row in g["table"]:
        acn = row["acn"]
        for t, w in enumerate(row["windows"]):
            first = 0 if acn < 0 else max(0, t - acn)
            assert w == sum(lens[first:t])                       # the chunks before t in the band, summed
            assert w == oracle.acn_window(starts, t, acn)
            st = np.asarray(starts, dtype=np.int64)
            assert w == vico.vico_acn_window(st, t, acn)       # the library's host-side rule


def exact_cos(u, v):
    """Cosine of two integer vectors whose norms are integers (3-4-5,
    5-12-13): an exact fraction; 0 for a zero vector."""
    dot = sum(a * b for a, b in zip(u, v))
    nu, nv = math.isqrt(sum(a * a for a in u)), math.isqrt(sum(b * b for b in v))
    assert nu * nu == sum(a * a for a in u) and nv * nv == sum(b * b for b in v)
    return Fraction(dot, nu * nv) if nu and nv else Fraction(0)


def test_drop_exact_cosines_fixture():
    g = load("drop_exact_cosines.json")
    vec, frames = g["vectors"], g["frames"]
    c, n_f = 3, len(frames[0])
    B = len(frames) // c
    for case in g["cases"]:
        tau = Fraction(str(case["tau"]))                     # the threshold as the decimal it is written as
        keep = np.ones((B, n_f), dtype=bool)
        smin = np.zeros((B, n_f))
        for b in range(B):
            for p in range(n_f):
                cos = [exact_cos(vec[frames[b * c + i][p]], vec[frames[b * c + j][p]])
                       for i in range(c) for j in range(i + 1, c)]
                keep[b, p] = not all(x > tau for x in cos)
                smin[b, p] = float(min(cos))
        index = [(b * c + f) * n_f + p for b in range(B) for f in range(c) for p in range(n_f)
                 if f == 0 or keep[b, p]]
        assert np.array_equal(np.asarray(case["keep"], dtype=bool), keep)
        assert case["index"] == index
        assert np.allclose(case["sim"], smin, rtol=0, atol=1e-15)
        # the oracle as it stands
        z = np.zeros((B, c, n_f, g["dm"]))
        for fi, row in enumerate(frames):
            for p, key in enumerate(row):
                z[fi // c, fi % c, p, :2] = vec[key]
        k2, s2, i2 = oracle.temporal_drop(z, case["tau"])
        assert np.array_equal(k2, keep) and i2.tolist() == index and np.allclose(s2, smin, rtol=0, atol=1e-15)
