"""Sustained streaming at the 3B layer shape: 64 chunks with ragged retained counts
(uniform in [256, 1024]), sink 64, W = R = 8192; per chunk the library attends
(history before the chunk, through the ring) and then appends.  Each chunk's
sampled rows are checked against the oracle run on the linear history, within
the derived per-element bounds of tests/_bounds.py."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_19849_amd as vico
from synth import ragged_chunk_lengths, stream_chunk, stream_sink
from tests._bounds import chunk_bound
from tests._gpu import check_bf16, dev

pytestmark = pytest.mark.gpu

Hq, Hkv, D, S, W, R = 16, 2, 128, 64, 8192, 8192


@pytest.mark.parametrize("window", [W, vico.VICO_FULL_HISTORY])
def test_stream_of_ragged_chunks(window):
    counts = ragged_chunk_lengths(64, 256, 1024, seed=0)
    ring_slots = R if window >= 0 else int(counts.sum())
    n_chunks = 64 if window >= 0 else 24
    sk_bits, sv_bits = stream_sink(S, Hkv, D, seed=0, family="F2")
    sk, sv = dev(sk_bits), dev(sv_bits)
    rk = torch.zeros((ring_slots, Hkv, D), dtype=torch.bfloat16, device="cuda")
    rv = torch.zeros_like(rk)
    sk64, sv64 = oracle.bf16_bits_to_f64(sk_bits), oracle.bf16_bits_to_f64(sv_bits)
    hist_k, hist_v = [], []
    H = 0
    rng = np.random.default_rng(5)
    starts = np.concatenate([[0], np.cumsum(counts)])
    wb = max(vico.vico_attn_plan(int(counts[t]), S, ring_slots, int(starts[t]), window, Hq, Hkv, D)[1]
             for t in range(n_chunks))
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
    for t in range(n_chunks):
        c = int(counts[t])
        qb, kb, vb = stream_chunk(t, c, Hq, Hkv, D, seed=0, family="F2")
        q, k, v = dev(qb), dev(kb), dev(vb)
        out = torch.empty((c, Hq, D), dtype=torch.bfloat16, device="cuda")
        lse = torch.empty((Hq, c), dtype=torch.float32, device="cuda")
        vico.vico_chunk_prefill_attn(q, k, v, sk, sv, rk, rv, H, window, out, lse=lse, workspace=ws)
        vico.vico_kv_append(k, v, rk, rv, H)
        rows = np.unique(np.concatenate([[0, c - 1], rng.choice(c, 6, replace=False)]))
        o = out[torch.from_numpy(rows).cuda()].float().cpu().numpy().astype(np.float64)
        l = lse[:, torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
        hk = np.concatenate(hist_k) if hist_k else np.zeros((0, Hkv, D))
        hv = np.concatenate(hist_v) if hist_v else np.zeros((0, Hkv, D))
        x = dict(q=oracle.bf16_bits_to_f64(qb), k_chunk=oracle.bf16_bits_to_f64(kb),
                 v_chunk=oracle.bf16_bits_to_f64(vb), sink_k=sk64, sink_v=sv64, hist_k=hk, hist_v=hv,
                 hist_len=H, window=window)
        ref, ref_lse = oracle.chunk_prefill_attention(**x, rows=rows)
        parts = vico.vico_attn_plan(c, S, ring_slots, H, window, Hq, Hkv, D)[0]
        b = chunk_bound(x, rows=rows, parts=parts)
        check_bf16(o, ref, b)
        assert np.all(np.abs(l - ref_lse) <= b.lse(ref_lse)), f"chunk {t}"
        hist_k.append(oracle.bf16_bits_to_f64(kb))
        hist_v.append(oracle.bf16_bits_to_f64(vb))
        if window >= 0 and sum(len(x) for x in hist_k) > 2 * W:      # keep the oracle's history short
            keep = np.concatenate(hist_k)[-W:], np.concatenate(hist_v)[-W:]
            hist_k, hist_v = [keep[0]], [keep[1]]
        H += c
    assert H > 4 * R or window < 0
