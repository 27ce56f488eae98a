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
