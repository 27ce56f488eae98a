"""Pins of the fp64 oracle against things other than itself.

Each test names what fixes the expected value: a library routine (torch's
scaled_dot_product_attention and bfloat16 conversion in float64 on the CPU),
a textbook special case (plain causal attention), a closed form, an
invariant, or brute force.  The mutation tests in test_oracle_mutants.py
check that planted mistakes in the oracle fail at least one of these.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle.attention import chunk_prefill_attention as attn, chunk_prefill_attention_rowloop as attn_rows
from synth import CONFIGS, ChunkShape, f32_to_bf16_bits, make_chunk_inputs, ragged_chunk_lengths
from tests._util import to_f64

SMALL_SHAPES = [
    CONFIGS["tiny"],
    CONFIGS["tiny_partial"],
    ChunkShape(7, 1, 16, 3, 64, 150, 37, 9),      # GQA 7:1, window < ring, ragged
    ChunkShape(4, 2, 8, 0, 32, 40, 0, 5),         # no sink, zero window
    ChunkShape(4, 4, 8, 2, 64, 50, -1, 7),        # full history, MHA
    ChunkShape(6, 2, 8, 5, 16, 0, 16, 4),         # empty history
    ChunkShape(2, 1, 8, 0, 8, 1000, 8, 1),        # one-row chunk, wrapped ring
]


def _sdpa_reference(x, shape):
    """torch SDPA (float64, CPU) over [sink | newest Wv history | chunk] with an explicit mask."""
    S, C = shape.sink_len, shape.chunk_len
    wv = shape.visible_window
    n = x["hist_k"].shape[0]
    k = np.concatenate([x["sink_k"], x["hist_k"][n - wv:], x["k_chunk"]], 0)
    v = np.concatenate([x["sink_v"], x["hist_v"][n - wv:], x["v_chunk"]], 0)
    mask = torch.ones(C, S + wv + C, dtype=torch.bool)
    mask[:, S + wv:] = torch.tril(torch.ones(C, C, dtype=torch.bool))
    qt = torch.from_numpy(x["q"]).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).permute(1, 0, 2)[None]
    vt = torch.from_numpy(v).permute(1, 0, 2)[None]
    o = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("shape", SMALL_SHAPES, ids=str)
@pytest.mark.parametrize("family", ["F1", "F2"])
def test_T1_blocked_equals_rowloop(shape, family):
    """T1: blocked dense form == per-row loop over explicitly listed keys."""
    x = to_f64(make_chunk_inputs(shape, seed=1, family=family))
    o1, l1 = attn(**x)
    o2, l2 = attn_rows(**x)
    assert np.max(np.abs(o1 - o2)) <= 1e-12
    assert np.max(np.abs(l1 - l2)) <= 1e-12


@pytest.mark.parametrize("shape", SMALL_SHAPES, ids=str)
@pytest.mark.parametrize("family", ["F1", "F2"])
def test_T2_matches_torch_sdpa(shape, family):
    """T2: library routine -- torch scaled_dot_product_attention in float64 with GQA."""
    x = to_f64(make_chunk_inputs(shape, seed=2, family=family))
    o, _ = attn(**x)
    ref = _sdpa_reference(x, shape)
    assert np.max(np.abs(o - ref)) <= 1e-12


@pytest.mark.parametrize("shape", [CONFIGS["tiny_partial"], ChunkShape(6, 3, 16, 4, 128, 90, 100, 12),
                                   ChunkShape(4, 1, 8, 2, 64, 30, 30, 10)], ids=str)
def test_T3_large_window_is_plain_causal_attention(shape):
    """T3: textbook case -- with W >= H the result is ordinary causal attention over
    the concatenated sequence [sink; history; chunk] (its last C rows), and equals
    full-history mode."""
    x = to_f64(make_chunk_inputs(shape, seed=3, family="F2"))
    o, lse = attn(**x)
    xf = dict(x, window=-1)
    of, lsef = attn(**xf)
    assert np.max(np.abs(o - of)) == 0.0 and np.max(np.abs(lse - lsef)) == 0.0
    seq_k = np.concatenate([x["sink_k"], x["hist_k"], x["k_chunk"]], 0)
    seq_v = np.concatenate([x["sink_v"], x["hist_v"], x["v_chunk"]], 0)
    L, C = seq_k.shape[0], shape.chunk_len
    Hq, Hkv = shape.num_q_heads, shape.num_kv_heads
    # queries for the prefix positions are irrelevant to the last C rows; use zeros
    seq_q = np.concatenate([np.zeros((L - C, Hq, shape.head_dim)), x["q"]], 0)
    t = lambda a: torch.from_numpy(a).permute(1, 0, 2)[None]
    ref = F.scaled_dot_product_attention(t(seq_q), t(seq_k), t(seq_v), is_causal=True, enable_gqa=True)
    ref = ref[0].permute(1, 0, 2).numpy()[L - C:]
    assert np.max(np.abs(o - ref)) <= 1e-12
    # log-sum-exp against torch.logsumexp of the same causal logits
    kk = torch.from_numpy(seq_k).repeat_interleave(Hq // Hkv, dim=1)        # [L, Hq, d]
    z = torch.einsum("chd,lhd->hcl", torch.from_numpy(x["q"]), kk) / math.sqrt(shape.head_dim)
    causal = torch.arange(L)[None, :] <= (torch.arange(C) + L - C)[:, None]
    ref_lse = torch.logsumexp(z.masked_fill(~causal[None], -math.inf), dim=-1).numpy()
    assert np.max(np.abs(lse - ref_lse)) <= 1e-12


@pytest.mark.parametrize("shape", SMALL_SHAPES, ids=str)
def test_T4_softmax_rows_sum_to_one(shape):
    """T4: with V == 1 everywhere each output equals the sum of the softmax weights: 1."""
    x = to_f64(make_chunk_inputs(shape, seed=4, family="F2"))
    for k in ("v_chunk", "sink_v", "hist_v"):
        x[k] = np.ones_like(x[k])
    o, _ = attn(**x)
    assert np.max(np.abs(o - 1.0)) <= 1e-12


@pytest.mark.parametrize("shape", [ChunkShape(2, 1, 64, 0, 256, 0, 256, 5),
                                   ChunkShape(4, 2, 128, 0, 64, 300, 0, 3)], ids=str)
def test_T5_single_visible_key(shape):
    """T5: row 0 with no sink and no visible history sees only chunk key 0:
    O equals V_0 exactly and LSE equals its single logit."""
    inp = make_chunk_inputs(shape, seed=5, family="F2")
    x = to_f64(inp)
    o, lse = attn(**x)
    g = shape.num_q_heads // shape.num_kv_heads
    for h in range(shape.num_q_heads):
        assert np.array_equal(o[0, h], x["v_chunk"][0, h // g])
        z0 = math.fsum(x["q"][0, h] * x["k_chunk"][0, h // g]) / math.sqrt(shape.head_dim)
        assert abs(lse[h, 0] - z0) <= 1e-15 * max(1.0, abs(z0))


def test_T6_ring_append_equals_linear_history():
    """T6: after appends the ring slot p mod R holds linear token p for the R newest p
    (bitwise), including wrap-around, for the tiny ring and a ragged stream."""
    for hist_len in (456, 200):
        R, C = 256, 64
        lin = np.arange((hist_len + C) * 3, dtype=np.int64).reshape(-1, 3)
        ring = oracle.RingModel.from_linear(lin[:hist_len], 0, R)
        H = ring.append(lin[hist_len:], hist_len)
        for p in range(max(0, H - R), H):
            assert np.array_equal(ring.buf[p % R], lin[p])
    R = 8192
    counts = ragged_chunk_lengths(64, 256, 1024, seed=0)
    lin = np.arange(int(counts.sum()), dtype=np.int64)[:, None]
    ring = oracle.RingModel(R, (1,), np.int64)
    H = 0
    for c in counts:
        H = ring.append(lin[H:H + c], H)
        lo = max(0, H - R)
        slots = np.arange(lo, H) % R
        assert np.array_equal(ring.buf[slots, 0], lin[lo:H, 0])
    assert H == counts.sum() and H > 4 * R


@pytest.mark.parametrize("R,H,W", [(256, 493, 250), (256, 456, 256), (256, 200, 256), (64, 1000, 37),
                                   (100, 100, 100), (16, 3, 16), (8192, 5 * 8192 + 777, 8192)])
def test_T7_window_gather_equals_linear_slice(R, H, W):
    """T7: reading the Wv newest tokens through ring slots (H - Wv + k) mod R gives
    lin[H - Wv : H] bitwise (window start straddling the wrap included)."""
    lin = np.arange(H * 2, dtype=np.int64).reshape(H, 2)
    ring = oracle.RingModel.from_linear(lin, 0, R)
    wv = oracle.visible_window(H, W)
    assert np.array_equal(ring.gather(H, wv), lin[H - wv:H])


def test_T8_lse_merge_of_disjoint_parts():
    """T8: attention over disjoint key subsets merged by log-sum-exp == attention over
    the union, including parts where some rows see no key at all."""
    rng = np.random.default_rng(8)
    n, L, d = 13, 97, 16
    q = rng.standard_normal((n, d)) * 2
    k = rng.standard_normal((L, d)) * 2
    v = rng.standard_normal((L, d))
    visible = rng.random((n, L)) < 0.7
    visible[:, 0] = True
    whole_o, whole_l = oracle.softmax_attention(q, k, v, visible, 0.25)
    for cuts in ([0, 30, 60, 97], [0, 1, 96, 97], [0, 50, 97], [0, 10, 20, 30, 40, 97]):
        outs, lses = [], []
        for a, b in zip(cuts[:-1], cuts[1:]):
            part = np.zeros_like(visible)
            part[:, a:b] = visible[:, a:b]
            o, l = oracle.softmax_attention(q, k, v, part, 0.25)
            outs.append(o); lses.append(l)
        mo, ml = oracle.lse_merge(outs, lses)
        assert np.max(np.abs(mo - whole_o)) <= 1e-12
        assert np.max(np.abs(ml - whole_l)) <= 1e-12
    # a row masked everywhere in one part
    part0 = np.zeros_like(visible); part0[1:, :40] = visible[1:, :40]
    part1 = np.zeros_like(visible); part1[:, 40:] = visible[:, 40:]; part1[0, :40] = visible[0, :40]
    o0, l0 = oracle.softmax_attention(q, k, v, part0, 0.25)
    o1, l1 = oracle.softmax_attention(q, k, v, part1, 0.25)
    assert l0[0] == -np.inf
    mo, ml = oracle.lse_merge([o0, o1], [l0, l1])
    assert np.max(np.abs(mo - whole_o)) <= 1e-12


@pytest.mark.parametrize("shape", SMALL_SHAPES[:3], ids=str)
def test_T9_constant_values_and_window_permutation(shape):
    """T9: V == c gives O == c; permuting the order of visible history tokens
    (all unmasked) leaves O and LSE unchanged."""
    x = to_f64(make_chunk_inputs(shape, seed=9, family="F2"))
    y = dict(x)
    for k in ("v_chunk", "sink_v", "hist_v"):
        y[k] = np.full_like(x[k], -0.3125)
    o, _ = attn(**y)
    assert np.max(np.abs(o + 0.3125)) <= 1e-13
    n, wv = x["hist_k"].shape[0], shape.visible_window
    perm = np.random.default_rng(9).permutation(wv)
    z = dict(x)
    z["hist_k"] = x["hist_k"].copy(); z["hist_v"] = x["hist_v"].copy()
    z["hist_k"][n - wv:] = x["hist_k"][n - wv:][perm]
    z["hist_v"][n - wv:] = x["hist_v"][n - wv:][perm]
    o1, l1 = attn(**x)
    o2, l2 = attn(**z)
    assert np.max(np.abs(o1 - o2)) <= 1e-13 and np.max(np.abs(l1 - l2)) <= 1e-12


def test_T10_linear_in_values():
    """T10: O(a V1 + b V2) == a O(V1) + b O(V2) for fixed Q, K."""
    sh = SMALL_SHAPES[2]
    x1 = to_f64(make_chunk_inputs(sh, seed=10, family="F2"))
    x2 = to_f64(make_chunk_inputs(sh, seed=11, family="F2"))
    a, b = 0.75, -1.5
    mix = dict(x1)
    for k in ("v_chunk", "sink_v", "hist_v"):
        mix[k] = a * x1[k] + b * x2[k]
    y2 = dict(x1)
    for k in ("v_chunk", "sink_v", "hist_v"):
        y2[k] = x2[k]
    o_mix, _ = attn(**mix)
    o1, _ = attn(**x1)
    o2, _ = attn(**y2)
    assert np.max(np.abs(o_mix - (a * o1 + b * o2))) <= 1e-12


def test_T11_large_logits_no_overflow_and_argmax_limit():
    """T11: logits scaled by 100 stay finite; when one visible key dominates by a wide
    margin, O equals that key's value to rounding."""
    sh = CONFIGS["tiny"]
    x = to_f64(make_chunk_inputs(sh, seed=12, family="F2"))
    x["q"] = x["q"] * 100.0
    o, lse = attn(**x)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    y = to_f64(make_chunk_inputs(sh, seed=13, family="F1"))
    # make sink key 3 align with every query of head 0/1 (one KV head) by a huge margin
    y["sink_k"][3, 0] = 0.0
    y["q"][:, :, :] = 0.0
    y["q"][:, :, 0] = 1.0
    y["sink_k"][3, 0, 0] = 4000.0
    o, lse = attn(**y)
    assert np.max(np.abs(o - y["sink_v"][3, 0][None, None, :])) <= 1e-12


@pytest.mark.parametrize("shape", SMALL_SHAPES, ids=str)
def test_T12_zero_query_closed_form(shape):
    """T12: closed form -- with Q == 0 all visible logits are equal, so row i averages
    exactly S + Wv + i + 1 values and LSE_i = log(S + Wv + i + 1)."""
    x = to_f64(make_chunk_inputs(shape, seed=14, family="F2"))
    x["q"] = np.zeros_like(x["q"])
    o, lse = attn(**x)
    S, C, wv = shape.sink_len, shape.chunk_len, shape.visible_window
    n = x["hist_v"].shape[0]
    g = shape.num_q_heads // shape.num_kv_heads
    for i in range(C):
        cnt = S + wv + i + 1
        assert np.max(np.abs(lse[:, i] - math.log(cnt))) <= 1e-13
        for h in range(shape.num_q_heads):
            kv = h // g
            tot = x["sink_v"][:, kv].sum(0) + x["hist_v"][n - wv:, kv].sum(0) + x["v_chunk"][:i + 1, kv].sum(0)
            assert np.max(np.abs(o[i, h] - tot / cnt)) <= 1e-13


def test_bf16_widening_matches_torch():
    """The oracle's bf16 widening agrees with torch's bfloat16 -> float64 conversion on
    every finite bit pattern."""
    bits = np.arange(65536, dtype=np.uint16)
    ours = oracle.bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    fin = np.isfinite(ref)
    assert np.array_equal(ours[fin], ref[fin])
    assert np.array_equal(np.isnan(ours), np.isnan(ref))


def test_synth_rounding_matches_torch_rne():
    """The generator's float32 -> bf16 rounding agrees with torch (round-to-nearest-even)."""
    x = np.random.default_rng(0).standard_normal(200000).astype(np.float32) * 3
    x[:4] = [1.00390625, 1.01171875, -1.00390625, 0.0]      # exact ties
    ours = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
