"""GPU parity of the bidirectional in-chunk option and of the chunk-granular
acn window (paper, Sec. 3 and the staircase mask of Eq. (4)) against the
oracle, whose readings are pinned to the literal mask in
test_oracle_acn_pins.py.  Tolerances: the derived per-element bounds of
tests/_bounds.py, as in test_gpu_parity.py."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_19849_amd as vico
from synth import make_chunk_inputs, ragged_chunk_lengths, stream_chunk, stream_sink
from tests._bounds import chunk_bound
from tests._gpu import DeviceChunk, check_bf16, check_f32, dev, oracle_and_bound
from tests.test_gpu_parity import SMALL

pytestmark = pytest.mark.gpu
BIDIR = vico.VICO_ATTN_BIDIRECTIONAL


@pytest.mark.parametrize("name", sorted(SMALL))
@pytest.mark.parametrize("splits", [0, 1, 3, -1])
def test_bidirectional_small_f2_fp32(name, splits):
    inp = make_chunk_inputs(SMALL[name], seed=301, family="F2")
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.float32, num_splits=splits, flags=BIDIR)
    ref, ref_lse, b = oracle_and_bound(inp, bidirectional=True, parts=dc.parts)
    check_f32(o, ref, b, lse, ref_lse)


@pytest.mark.parametrize("name", ["tiny", "gqa7_ragged", "balanced_many_parts"])
def test_bidirectional_bf16(name):
    inp = make_chunk_inputs(SMALL[name], seed=302, family="F2")
    dc = DeviceChunk(inp)
    o, _ = dc.attention(torch.bfloat16, flags=BIDIR)
    ref, _, b = oracle_and_bound(inp, bidirectional=True, parts=dc.parts)
    check_bf16(o, ref, b)


@pytest.mark.parametrize("cfg", ["7b_wrap", "3b_wrap"])
def test_bidirectional_full_size_sampled_rows(cfg):
    """Full 7B/3B-shaped chunk with every row seeing the whole chunk: all row
    tiles then share one key count (the schedule differs from the causal one),
    sampled rows of every row tile against the oracle, bf16 output and LSE."""
    from synth import CONFIGS
    sh = CONFIGS[cfg]
    inp = make_chunk_inputs(sh, seed=5, family="F2")
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.bfloat16, flags=BIDIR)
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([rng.choice(sh.chunk_len, 24, replace=False),
                                     [0, 255, 256, sh.chunk_len - 1]]))
    ref, ref_lse, b = oracle_and_bound(inp, rows=rows, bidirectional=True, parts=dc.parts)
    check_bf16(o[rows], ref, b)
    assert np.all(np.abs(lse[:, rows] - ref_lse) <= b.lse(ref_lse))


@pytest.mark.parametrize("flags", [0, BIDIR])
def test_acn_window_stream(flags):
    """32 ragged chunks (256..1024 tokens) at 3B heads with the window set to
    the 4 most recent whole chunks; the ring holds 4 * 1024 slots, so the
    window read wraps; attend then append per chunk."""
    Hq, Hkv, D, S, acn, R = 16, 2, 128, 64, 4, 4096
    counts = ragged_chunk_lengths(32, 256, 1024, seed=3)
    starts = np.concatenate([[0], np.cumsum(counts)])
    sk_bits, sv_bits = stream_sink(S, Hkv, D, seed=3, family="F2")
    sk, sv = dev(sk_bits), dev(sv_bits)
    rk = torch.zeros((R, Hkv, D), dtype=torch.bfloat16, device="cuda")
    rv = torch.zeros_like(rk)
    sk64, sv64 = oracle.bf16_bits_to_f64(sk_bits), oracle.bf16_bits_to_f64(sv_bits)
    hk_all, hv_all = [], []
    rng = np.random.default_rng(7)
    ws = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    for t, c in enumerate(counts):
        c = int(c)
        H = int(starts[t])
        W = vico.vico_acn_window(list(starts[:t + 1]), t, acn)
        assert W == oracle.acn_window(starts, t, acn)
        qb, kb, vb = stream_chunk(t, c, Hq, Hkv, D, seed=3, family="F2")
        q, k, v = dev(qb), dev(kb), dev(vb)
        out = torch.empty((c, Hq, D), dtype=torch.float32, device="cuda")
        lse = torch.empty((Hq, c), dtype=torch.float32, device="cuda")
        assert vico.vico_attn_plan(c, S, R, H, W, Hq, Hkv, D, 0, flags)[1] <= ws.numel()
        vico.vico_chunk_prefill_attn(q, k, v, sk, sv, rk, rv, H, W, out, lse=lse, workspace=ws, flags=flags)
        vico.vico_kv_append(k, v, rk, rv, H)
        rows = np.unique(np.concatenate([[0, c - 1], rng.choice(c, 8, replace=False)]))
        o = out[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
        l = lse[:, torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
        hk = np.concatenate(hk_all) if hk_all else np.zeros((0, Hkv, D))
        hv = np.concatenate(hv_all) if hv_all else np.zeros((0, Hkv, D))
        x = dict(q=oracle.bf16_bits_to_f64(qb), k_chunk=oracle.bf16_bits_to_f64(kb),
                 v_chunk=oracle.bf16_bits_to_f64(vb), sink_k=sk64, sink_v=sv64, hist_k=hk, hist_v=hv,
                 hist_len=H, window=W)
        ref, ref_lse = oracle.chunk_prefill_attention(**x, rows=rows, bidirectional=bool(flags & BIDIR))
        parts = vico.vico_attn_plan(c, S, R, H, W, Hq, Hkv, D, 0, flags)[0]
        b = chunk_bound(x, rows=rows, bidirectional=bool(flags & BIDIR), parts=parts)
        check_f32(o, ref, b, l, ref_lse)
        hk_all.append(oracle.bf16_bits_to_f64(kb))
        hv_all.append(oracle.bf16_bits_to_f64(vb))
        if len(hk_all) > acn + 1:
            hk_all, hv_all = hk_all[1:], hv_all[1:]
