"""GPU parity of the ring-buffer append (bit-exact against the oracle's ring model)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_19849_amd as vico
from synth import f32_to_bf16_bits, ragged_chunk_lengths
from tests._gpu import bits_of, dev

pytestmark = pytest.mark.gpu


def _rand_bits(rng, shape):
    return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


@pytest.mark.parametrize("R,H,C,Hkv,D", [
    (256, 456, 64, 1, 64),          # tiny ring, write pointer 200: no wrap
    (256, 200, 64, 1, 64),          # partial history: evicts nothing yet, wraps past 255
    (256, 250, 64, 1, 64),          # wraps after 6 tokens
    (100, 37, 100, 2, 128),         # chunk as long as the ring
    (16384, 5 * 16384 + 777, 2048, 4, 128),
    (16384, 16384 - 100, 2048, 4, 128),
    (8192, 0, 1, 2, 128),
])
def test_append_matches_ring_model(R, H, C, Hkv, D):
    rng = np.random.default_rng(R + H + C)
    ring0 = _rand_bits(rng, (R, Hkv, D))
    k, v = _rand_bits(rng, (C, Hkv, D)), _rand_bits(rng, (C, Hkv, D))
    rk, rv = dev(ring0), dev(ring0.copy())
    vico.vico_kv_append(dev(k), dev(v), rk, rv, H)
    torch.cuda.synchronize()
    mk, mv = oracle.RingModel(R, (Hkv, D)), oracle.RingModel(R, (Hkv, D))
    mk.buf[:] = ring0
    mv.buf[:] = ring0
    mk.append(k, H)
    mv.append(v, H)
    assert np.array_equal(bits_of(rk), mk.buf)
    assert np.array_equal(bits_of(rv), mv.buf)


def test_ragged_stream_of_appends():
    """64 appends of ragged lengths (256..1024) into an 8192-slot ring: after every
    append the device ring equals the model, and the newest R tokens sit at p mod R."""
    R, Hkv, D = 8192, 2, 128
    counts = ragged_chunk_lengths(64, 256, 1024, seed=0)
    rng = np.random.default_rng(7)
    rk = torch.zeros((R, Hkv, D), dtype=torch.bfloat16, device="cuda")
    rv = torch.zeros_like(rk)
    mk, mv = oracle.RingModel(R, (Hkv, D)), oracle.RingModel(R, (Hkv, D))
    H = 0
    lin_k = []
    for t, c in enumerate(counts):
        k, v = _rand_bits(rng, (c, Hkv, D)), _rand_bits(rng, (c, Hkv, D))
        lin_k.append(k)
        vico.vico_kv_append(dev(k), dev(v), rk, rv, H)
        mk.append(k, H)
        mv.append(v, H)
        H += int(c)
        if t % 8 == 7 or t == len(counts) - 1:
            torch.cuda.synchronize()
            assert np.array_equal(bits_of(rk), mk.buf), f"K ring differs after chunk {t}"
            assert np.array_equal(bits_of(rv), mv.buf), f"V ring differs after chunk {t}"
    lin = np.concatenate(lin_k)
    got = bits_of(rk)
    assert np.array_equal(got[np.arange(H - R, H) % R], lin[H - R:H])


@pytest.mark.parametrize("splits,flags", [(0, 0), (1, 0), (4, 0), (12, 0), (0, vico.VICO_ATTN_BIDIRECTIONAL)])
def test_attention_with_append_equals_attention_then_append(splits, flags):
    """VICO_ATTN_APPEND: one call attends and then appends (the copy rides on
    the split merge, or runs as its own launch without a split).  Over a
    stream of ragged chunks through a ring that wraps, outputs, LSE and the
    ring must equal, bit for bit, an attention call followed by
    vico_kv_append on a second ring; the ring must also equal the oracle's
    ring model."""
    Hq, Hkv, D, S, R, W = 8, 2, 128, 16, 1024, 1024
    rng = np.random.default_rng(70 + splits + flags)
    counts = [300, 513, 64, 1000, 1024, 7, 700]
    sk, sv = dev(_rand_bits(rng, (S, Hkv, D))), dev(_rand_bits(rng, (S, Hkv, D)))
    ring0 = _rand_bits(rng, (R, Hkv, D))
    rk_a, rv_a = dev(ring0), dev(ring0.copy())
    rk_b, rv_b = dev(ring0.copy()), dev(ring0.copy())
    mk, mv = oracle.RingModel(R, (Hkv, D)), oracle.RingModel(R, (Hkv, D))
    mk.buf[:] = ring0
    mv.buf[:] = ring0
    ws = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    H = 5 * R + 333
    for c in counts:
        qb, kb, vb = (_rand_bits(rng, (c, Hq, D)), _rand_bits(rng, (c, Hkv, D)), _rand_bits(rng, (c, Hkv, D)))
        q, k, v = dev(qb), dev(kb), dev(vb)
        outs = []
        for rk, rv, fl in ((rk_a, rv_a, flags), (rk_b, rv_b, flags | vico.VICO_ATTN_APPEND)):
            out = torch.empty((c, Hq, D), dtype=torch.float32, device="cuda")
            lse = torch.empty((Hq, c), dtype=torch.float32, device="cuda")
            assert vico.vico_attn_plan(c, S, R, H, W, Hq, Hkv, D, splits, fl)[1] <= ws.numel()
            vico.vico_chunk_prefill_attn(q, k, v, sk, sv, rk, rv, H, W, out, lse=lse, workspace=ws,
                                         num_splits=splits, flags=fl)
            if not fl & vico.VICO_ATTN_APPEND:
                vico.vico_kv_append(k, v, rk, rv, H)
            outs.append((out, lse))
        torch.cuda.synchronize()
        assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
        assert torch.equal(rk_a, rk_b) and torch.equal(rv_a, rv_b)
        mk.append(kb, H)
        mv.append(vb, H)
        assert np.array_equal(bits_of(rk_b), mk.buf) and np.array_equal(bits_of(rv_b), mv.buf)
        H += c


@pytest.mark.parametrize("C,splits", [(300, 0), (513, 3), (1024, 0)])
def test_chunk_call_with_append_replays_as_a_graph(C, splits):
    """A chunk call with VICO_ATTN_APPEND (attention, the split merge and the
    ring copy riding on it; a 300-token chunk runs the packed row tiles)
    captured into a HIP graph replays the eager result bit for bit, replay
    after replay, with an eager call of another window on the same buffers in
    between.  The window and the appended slots do not overlap (W + C <= R),
    so every replay sees the same window and writes the same slots."""
    Hq, Hkv, D, S, R, W, W2 = 8, 2, 128, 16, 2048, 900, 300
    assert W + C <= R
    rng = np.random.default_rng(C + splits)
    sk, sv = dev(_rand_bits(rng, (S, Hkv, D))), dev(_rand_bits(rng, (S, Hkv, D)))
    ring0 = _rand_bits(rng, (R, Hkv, D))
    rk, rv = dev(ring0), dev(ring0.copy())
    q, k, v = (dev(_rand_bits(rng, (C, Hq, D))), dev(_rand_bits(rng, (C, Hkv, D))),
               dev(_rand_bits(rng, (C, Hkv, D))))
    H = 3 * R + 555
    parts, wb = vico.vico_attn_plan(C, S, R, H, W, Hq, Hkv, D, splits, vico.VICO_ATTN_APPEND)
    assert parts > 1                  # the merge (and the append on it) is part of the graph
    ws = torch.empty(max(wb, vico.vico_attn_plan(C, S, R, H, W2, Hq, Hkv, D)[1]), dtype=torch.uint8, device="cuda")
    out = torch.empty((C, Hq, D), dtype=torch.float32, device="cuda")
    lse = torch.empty((Hq, C), dtype=torch.float32, device="cuda")

    def call(window, flags):
        vico.vico_chunk_prefill_attn(q, k, v, sk, sv, rk, rv, H, window, out, lse=lse, workspace=ws,
                                     num_splits=splits if window == W else 0, flags=flags)

    call(W, vico.VICO_ATTN_APPEND)
    torch.cuda.synchronize()
    eager = (out.clone(), lse.clone(), rk.clone(), rv.clone())
    mk = oracle.RingModel(R, (Hkv, D))
    mk.buf[:] = ring0
    mk.append(bits_of(k), H)
    assert np.array_equal(bits_of(rk), mk.buf)
    call(W2, 0)
    torch.cuda.synchronize()
    other = (out.clone(), lse.clone())

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        call(W, vico.VICO_ATTN_APPEND)        # warm-up on the capture stream
        torch.cuda.current_stream().synchronize()
        with torch.cuda.graph(graph, stream=side):
            call(W, vico.VICO_ATTN_APPEND)
    torch.cuda.synchronize()
    for _ in range(3):
        call(W2, 0)                           # eager call of another window, same buffers
        torch.cuda.synchronize()
        assert torch.equal(out, other[0]) and torch.equal(lse, other[1])
        out.zero_()
        lse.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager[0]) and torch.equal(lse, eager[1])
        assert torch.equal(rk, eager[2]) and torch.equal(rv, eager[3])
