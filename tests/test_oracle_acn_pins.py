"""Pins of the chunk-granular window and the bidirectional option against the
additive mask of Eq. (4) written out token by token (paper, Sec. 3: the
vision rows of chunk t see the chunks t-acn .. t -- a staircase band).

The whole stream (sink prefix, then ragged visual chunks) is one sequence;
torch's scaled_dot_product_attention in float64 with that explicit mask is
the reference, and every chunk's rows must equal the bounded chunk prefill
with window = acn_window(...)."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
from synth import stream_chunk, stream_sink

f64 = oracle.bf16_bits_to_f64


def _stream(n_chunks, Hq, Hkv, D, S, seed, lo=3, hi=40):
    lens = np.random.default_rng(seed).integers(lo, hi + 1, n_chunks)
    chunks = [tuple(f64(x) for x in stream_chunk(t, int(c), Hq, Hkv, D, seed=seed, family="F2"))
              for t, c in enumerate(lens)]
    sk, sv = (f64(x) for x in stream_sink(S, Hkv, D, seed=seed, family="F2"))
    return lens, chunks, sk, sv


def _eq4_reference(lens, chunks, sk, sv, acn, causal):
    """Attention of every vision token over the whole stream under the mask of
    Eq. (4): token i of chunk t sees sink tokens and token j of chunk u iff
    t - acn <= u <= t (acn < 0: u <= t), and with `causal` also j <= i."""
    S = sk.shape[0]
    q = np.concatenate([c[0] for c in chunks])
    k = np.concatenate([sk] + [c[1] for c in chunks])
    v = np.concatenate([sv] + [c[2] for c in chunks])
    chunk_of = np.concatenate([np.full(int(c), t) for t, c in enumerate(lens)])
    n = len(chunk_of)
    mask = np.zeros((n, S + n), dtype=bool)
    mask[:, :S] = True
    for i in range(n):
        t = chunk_of[i]
        for j in range(n):
            u = chunk_of[j]
            ok = (u <= t) and (acn < 0 or u >= t - acn)
            if causal:
                ok = ok and j <= i
            mask[i, S + j] = ok
    Hq, Hkv = q.shape[1], k.shape[1]
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2)[None]
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=torch.from_numpy(mask),
                                                           enable_gqa=True)[0].permute(1, 0, 2).numpy()
    g = Hq // Hkv
    z = torch.einsum("nhd,lhd->hnl", torch.from_numpy(q), torch.from_numpy(k).repeat_interleave(g, dim=1))
    z = z / math.sqrt(q.shape[2])
    lse = torch.logsumexp(z.masked_fill(~torch.from_numpy(mask)[None], -math.inf), dim=-1).numpy()
    return out, lse


@pytest.mark.parametrize("acn", [0, 1, 2, 5, -1])
@pytest.mark.parametrize("causal", [True, False])
def test_chunk_prefill_with_acn_window_equals_eq4_mask(acn, causal):
    Hq, Hkv, D, S = 4, 2, 16, 3
    lens, chunks, sk, sv = _stream(9, Hq, Hkv, D, S, seed=acn + 10)
    ref_o, ref_l = _eq4_reference(lens, chunks, sk, sv, acn, causal)
    starts = np.concatenate([[0], np.cumsum(lens)])
    hk = np.concatenate([c[1] for c in chunks])
    hv = np.concatenate([c[2] for c in chunks])
    for t, c in enumerate(lens):
        H = int(starts[t])
        W = oracle.acn_window(starts, t, acn)
        q, kc, vc = chunks[t]
        o, l = oracle.chunk_prefill_attention(q, kc, vc, sk, sv, hk[:H], hv[:H], H, W, bidirectional=not causal)
        np.testing.assert_allclose(o, ref_o[H:H + c], rtol=0, atol=1e-12)
        np.testing.assert_allclose(l, ref_l[:, H:H + c], rtol=0, atol=1e-12)


def test_acn_window_closed_forms():
    starts = np.array([0, 10, 25, 40, 70, 71])
    assert oracle.acn_window(starts, 0, 3) == 0                 # first chunk: no history
    assert oracle.acn_window(starts, 2, 5) == 25                # fewer than acn chunks before: all
    assert oracle.acn_window(starts, 4, 0) == 0                 # acn = 0: the chunk alone
    assert oracle.acn_window(starts, 4, 1) == 30                # exactly the previous chunk
    assert oracle.acn_window(starts, 5, 2) == 31
    assert oracle.acn_window(starts, 5, -1) == 71               # unbounded


def test_bidirectional_full_history_is_unmasked_attention():
    """Window >= history and no causal mask: plain softmax attention of the
    chunk rows over [sink | history | chunk], every key visible."""
    Hq, Hkv, D, S = 2, 1, 8, 2
    lens, chunks, sk, sv = _stream(3, Hq, Hkv, D, S, seed=4)
    hk = np.concatenate([c[1] for c in chunks[:2]])
    hv = np.concatenate([c[2] for c in chunks[:2]])
    q, kc, vc = chunks[2]
    o, _ = oracle.chunk_prefill_attention(q, kc, vc, sk, sv, hk, hv, hk.shape[0], -1, bidirectional=True)
    k = np.concatenate([sk, hk, kc])[:, 0]
    v = np.concatenate([sv, hv, vc])[:, 0]
    for h in range(Hq):
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q[:, h])[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None])[0].numpy()
        np.testing.assert_allclose(o[:, h], ref, rtol=0, atol=1e-12)


def test_bidirectional_rows_of_a_chunk_share_their_keys():
    """Without the causal mask every row of the chunk sees the same key set:
    with Q = 0 all rows give the same output and LSE = log(S + Wv + C)."""
    Hq, Hkv, D, S = 2, 1, 8, 2
    lens, chunks, sk, sv = _stream(2, Hq, Hkv, D, S, seed=5)
    hk, hv = chunks[0][1], chunks[0][2]
    q, kc, vc = chunks[1]
    o, l = oracle.chunk_prefill_attention(np.zeros_like(q), kc, vc, sk, sv, hk, hv, hk.shape[0], 7,
                                          bidirectional=True)
    assert np.allclose(o, o[:1], atol=1e-15)
    np.testing.assert_allclose(l, math.log(S + min(7, hk.shape[0]) + q.shape[0]), atol=1e-13)
