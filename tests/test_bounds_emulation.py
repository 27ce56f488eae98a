"""The derived GPU tolerance (tests/_bounds.py) against an emulation of the
kernels' arithmetic on the CPU.

The emulation runs the online softmax of the attention kernels in float32
with bf16-rounded probabilities for the P.V product: 32-key halves,
exponentials against the running max first, the max raised (O and l
rescaled, the half redone) only when a 16-key lane sum exceeds 2^8 or the row
has no max yet.  For rows of given fp32 logits and bf16 values it must stay
inside the per-element bound, and plausible slips in that arithmetic must
leave it: the bound is tight enough to see them.  Logit patterns: uniform
(the literal N(0,1)/sqrt(d) workload), logits of std 4, near one-hot rows,
and a jump of the row max by just over 2^8 while many earlier keys still
carry most of the weight (the case where a wrong rescale factor matters).
"""
import math

import numpy as np
import pytest

from synth import f32_to_bf16_bits
from oracle import bf16_bits_to_f64
from oracle.attention import default_scale
import oracle
from tests._bounds import Bound, U8, U24

LOG2E = 1.0 / math.log(2.0)


def bf16(x):
    return bf16_bits_to_f64(f32_to_bf16_bits(np.asarray(x, np.float32))).astype(np.float32)


def bf16_truncate(x):
    b = np.asarray(x, np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
    return b.view(np.float32)


def emulate(s, V, scale, slip=None):
    """One row: fp32 logits s [L], values V [L, d] (bf16 values) -> fp32 O [d]."""
    c = np.float32(scale * LOG2E)
    s = s.astype(np.float32)
    m, l = np.float32(-np.inf), np.float32(0.0)
    o = np.zeros(V.shape[1], np.float32)
    rnd = bf16_truncate if slip == "truncate" else bf16
    for h0 in range(0, len(s), 32):
        sh = s[h0:h0 + 32]
        vh = V[h0:h0 + 32].astype(np.float32)

        def expo(m_):
            neg = np.float32(0.0) if m_ == -np.inf else -m_
            return np.exp2((sh * c + neg).astype(np.float32)).astype(np.float32)

        p = expo(m)
        lanes = [p[i:i + 16].sum(dtype=np.float32) for i in range(0, len(p), 16)]
        if m == -np.inf or max(lanes) > 256.0:
            m_new = np.float32(max(m, np.float32(sh.max()) * c))
            alpha = np.float32(1.0) if m_new == m else np.float32(np.exp2(m - m_new))
            if slip == "alpha" and m != -np.inf:
                alpha = np.float32(alpha * 1.03)
            if slip != "forget_l":
                l = np.float32(l * alpha)
            o = (o * alpha).astype(np.float32)
            m = m_new
            p = expo(m)
        l = np.float32(l + p.sum(dtype=np.float32))
        o = (o + rnd(p) @ vh).astype(np.float32)
    return o / l


def exact(s, V):
    s = s.astype(np.float64)
    p = np.exp(s - s.max())
    l = p.sum()
    return p @ V / l, p @ np.abs(V) / l


def rows(kind, rng, L=2000, d=64):
    """(logits, values, scale) of one row; logits are fp32 values, values bf16."""
    scale = 1.0 / math.sqrt(d)
    V = bf16(rng.standard_normal((L, d)))
    if kind == "uniform":        # N(0,1)/sqrt(d) inputs: logits of std ~1/d
        s = rng.standard_normal(L) / d
    elif kind == "std4":         # logits of std 4 (F2)
        s = rng.standard_normal(L) * 4.0 / scale
    elif kind == "peaked":       # nearly one-hot
        s = rng.standard_normal(L) * 20.0 / scale
    elif kind == "jump":
        # Many earlier keys near the running max carry ~3/4 of the weight when
        # one key lands 8.4 (log2) above them and forces a rescale; the values
        # of the two groups differ, so the rescale factor shows in O.
        s = rng.standard_normal(L) * 0.05 / scale
        j = 1000 + int(rng.integers(0, 500))
        s[j] = (s[:j].max() * scale * LOG2E + 8.4) / (scale * LOG2E)
        s[j + 1:] = -40.0 / scale
        V = bf16(1.0 + 0.1 * rng.standard_normal((L, d)))
        V[j] = bf16(-1.0 + 0.1 * rng.standard_normal(d))
    else:
        raise ValueError(kind)
    return bf16(s).astype(np.float32), V, scale


def bound_for(s, V, scale, A, ref):
    # logits are exact fp32 inputs here: only the scaling, the FMA and exp2 round
    zmax = np.max(np.abs(s.astype(np.float64))) * scale
    dz = zmax * 3 * U24 + 128 * U24
    b = Bound(A[None, None, :], np.array([[dz + 2.0 ** -22]]), np.array([[dz]]), len(s))
    return b.f32(ref[None, None, :])[0, 0]


KINDS = ["uniform", "std4", "peaked", "jump"]


@pytest.mark.parametrize("kind", KINDS)
def test_emulated_kernel_arithmetic_stays_inside_the_bound(kind):
    rng = np.random.default_rng(KINDS.index(kind))
    for _ in range(12):
        s, V, scale = rows(kind, rng)
        ref, A = exact(s.astype(np.float64) * scale, V.astype(np.float64))
        got = emulate(s, V, scale).astype(np.float64)
        assert np.all(np.abs(got - ref) <= bound_for(s, V, scale, A, ref))


@pytest.mark.parametrize("slip,kind", [("alpha", "jump"), ("truncate", "peaked"), ("forget_l", "jump")])
def test_planted_slips_leave_the_bound(slip, kind):
    """A rescale factor off by 3 %, probabilities truncated to bf16 instead of
    rounded to nearest even, and a rescale that forgets l: each exceeds the
    bound on some row of the pattern that exposes it."""
    rng = np.random.default_rng(100 + KINDS.index(kind))
    hit = False
    for _ in range(12):
        s, V, scale = rows(kind, rng)
        ref, A = exact(s.astype(np.float64) * scale, V.astype(np.float64))
        got = emulate(s, V, scale, slip=slip).astype(np.float64)
        hit |= bool(np.any(np.abs(got - ref) > bound_for(s, V, scale, A, ref)))
    assert hit


def test_bound_is_within_a_small_factor_of_the_bf16_unit():
    """Sanity of the scale: on near one-hot rows of 2000 keys the worst-case
    bound is below 1.5 u8 times sum p|v|/l, and the observed error uses a good
    part of it on some element (the bound is not loose by orders of
    magnitude)."""
    rng = np.random.default_rng(7)
    ratio = 0.0
    for _ in range(12):
        s, V, scale = rows("peaked", rng)
        ref, A = exact(s.astype(np.float64) * scale, V.astype(np.float64))
        b = bound_for(s, V, scale, A, ref)
        assert np.all(b <= 1.5 * U8 * A + 1e-30)
        got = emulate(s, V, scale).astype(np.float64)
        ratio = max(ratio, float(np.max(np.abs(got - ref) / b)))
    assert ratio > 0.2


def _emulate_rows(q, keys, vals, visible, scale):
    """Emulated kernel over a [Lq, L] visibility mask for one head; fp32 logits
    from bf16 inputs (fp32 products and sums)."""
    s_all = keys.astype(np.float32) @ q.astype(np.float32).T            # [L, Lq] fp32
    out = np.zeros((q.shape[0], vals.shape[1]))
    for i in range(q.shape[0]):
        idx = np.flatnonzero(visible[i])
        out[i] = emulate(s_all[idx, i], vals[idx].astype(np.float32), scale)
    return out


@pytest.mark.parametrize("family", ["F1", "F2"])
def test_chunk_bound_holds_for_the_emulated_kernel(family):
    """chunk_bound on a whole tiny chunk prefill (sink, a wrapped window of
    history, causal chunk) covers the emulated kernel on every element."""
    from synth import CONFIGS, make_chunk_inputs
    from tests._bounds import chunk_bound
    from tests._util import to_f64
    inp = make_chunk_inputs(CONFIGS["tiny"], seed=3, family=family)
    x = to_f64(inp)
    C, Hq, d = x["q"].shape
    Hkv = x["k_chunk"].shape[1]
    ref, _ = oracle.chunk_prefill_attention(**x)
    b = chunk_bound(x)
    wv = oracle.visible_window(x["hist_len"], x["window"])
    n = x["hist_k"].shape[0]
    S = x["sink_k"].shape[0]
    vis = np.ones((C, S + wv + C), bool)
    vis[:, S + wv:] = np.tril(np.ones((C, C), bool))
    for h in range(Hq):
        kv = h // (Hq // Hkv)
        keys = np.concatenate([x["sink_k"][:, kv], x["hist_k"][n - wv:n, kv], x["k_chunk"][:, kv]])
        vals = np.concatenate([x["sink_v"][:, kv], x["hist_v"][n - wv:n, kv], x["v_chunk"][:, kv]])
        got = _emulate_rows(x["q"][:, h], keys, vals, vis, default_scale(d))
        assert np.all(np.abs(got - ref[:, h]) <= b.f32(ref)[:, h])


def test_gather_bound_holds_for_the_emulated_kernel():
    from synth import QUERY_CONFIGS, make_query_inputs
    from tests._bounds import gather_bound
    qi = make_query_inputs(QUERY_CONFIGS["q_small"], seed=11, family="F2")
    sh = qi.shape
    k, v = qi.store_kv()
    sel = oracle.select_chunks(np.random.default_rng(1).uniform(size=sh.num_chunks), sh.top_k)
    st, ln = oracle.chunk_segments(sel, qi.chunk_start, qi.chunk_len)
    f = bf16_bits_to_f64
    args = (f(qi.q), f(qi.tail_k), f(qi.tail_v), f(qi.sink_k), f(qi.sink_v), f(k), f(v), st, ln)
    ref, _ = oracle.gather_attention(*args)
    b = gather_bound(*args)
    Lq, Hq, d = args[0].shape
    T, S = sh.tail_len, sh.sink_len
    G = int(np.sum(ln))
    vis = np.ones((Lq, S + G + T), bool)
    vis[:, S + G:] = np.arange(T)[None, :] <= (T - Lq + np.arange(Lq))[:, None]
    for h in range(Hq):
        kv = h // (Hq // sh.num_kv_heads)
        seg = lambda a: np.concatenate([a[s0:s0 + m, kv] for s0, m in zip(st, ln)])
        keys = np.concatenate([args[3][:, kv], seg(args[5]), args[1][:, kv]])
        vals = np.concatenate([args[4][:, kv], seg(args[6]), args[2][:, kv]])
        got = _emulate_rows(args[0][:, h], keys, vals, vis, default_scale(d))
        assert np.all(np.abs(got - ref[:, h]) <= b.f32(ref)[:, h])
