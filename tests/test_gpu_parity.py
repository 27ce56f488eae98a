"""GPU parity: the HIP attention path against the fp64 oracle, element by element.

Small shapes are compared in full; the full-size workloads (3B/7B layer
shapes, full-history 65536 tokens) run the whole chunk on the GPU in the
launch configuration the benchmark times and are compared on sampled rows.

Tolerances (derived in tests/_bounds.py from the kernels' arithmetic and
pinned against an emulation of it in tests/test_bounds_emulation.py)
  * every element: |O_gpu - O| <= (2^-8 + 2 eta + kappa) * sum_j p_j |v_j| / l
    (bf16 rounding of the probabilities, fp32 logits, fp32 accumulation),
    plus half a bf16 ulp for bf16 output; sum_j p_j |v_j| / l is the oracle's
    attention over |V|; the LSE within the largest logit error plus fp32
    rounding;
  * F2U inputs (Q, K ~ 2 N(0,1), V uniform in [-1, 1], so |O| <= 1): also the
    stated gate read literally, max-abs <= 1e-2 and mean-abs <= 1e-3;
  * F1 inputs (N(0,1)/sqrt(d), outputs ~1e-3): also the per-element Hoeffding
    bound of the bf16 rounding noise and the relative Frobenius error
    <= 5e-3; the errors normalised by rms(O) are reported;
  * integer-valued Q and K (large logits, rising maxima): every dot product is
    exact in fp32, so the bound is the bf16 unit almost alone.
"""
import numpy as np
import pytest
import torch

import paper_2606_19849_amd as vico
from oracle import bf16_bits_to_f64
from synth import CONFIGS, ChunkShape, f32_to_bf16_bits, make_chunk_inputs
from tests._gpu import (DeviceChunk, check_bf16, check_f1, check_f32, check_literal, check_relative,
                        oracle_and_bound, oracle_result)

pytestmark = pytest.mark.gpu

SMALL = {
    "tiny": CONFIGS["tiny"],
    "tiny_partial": CONFIGS["tiny_partial"],
    "gqa7_ragged": ChunkShape(14, 2, 128, 5, 700, 1333, 600, 300),
    "wrap_midtile": ChunkShape(4, 1, 128, 5, 256, 868, 250, 131),
    "full_mode": ChunkShape(4, 2, 128, 7, 512, 400, -1, 77),
    "no_sink_no_hist": ChunkShape(2, 2, 128, 0, 0, 0, 0, 150),
    "window0": ChunkShape(4, 1, 64, 3, 64, 500, 0, 70),
    "one_row": ChunkShape(8, 2, 128, 64, 1024, 5000, 1000, 1),
    "mha_d64": ChunkShape(3, 3, 64, 9, 300, 299, 300, 257),
    "auto_split": ChunkShape(2, 1, 128, 64, 4096, 4096, 4096, 200),
    # enough key tiles for the balanced schedule (>= 4 per work-group); row tiles
    # spread over many work-groups, ring read wrapping
    "balanced_many_parts": ChunkShape(8, 2, 128, 64, 4096, 4596, 4000, 600),
    "balanced_d64": ChunkShape(4, 1, 64, 16, 8192, 10000, 8000, 300),
    # many heads: 168 and 144 (row tile, head) pairs, between half and all of
    # the work-groups; ring read wrapping
    "many_heads": ChunkShape(56, 8, 128, 16, 640, 900, 512, 520),
    "many_heads_d64": ChunkShape(48, 6, 64, 9, 300, 777, 300, 700),
}


@pytest.mark.parametrize("name", sorted(SMALL))
@pytest.mark.parametrize("splits", [0, 1, 3, -1])
def test_small_f2_fp32(name, splits):
    inp = make_chunk_inputs(SMALL[name], seed=101, family="F2")
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.float32, num_splits=splits)
    ref, ref_lse, b = oracle_and_bound(inp, parts=dc.parts)
    check_f32(o, ref, b, lse, ref_lse)


def _ragged_gqa_shapes(n=12, seed=2024):
    """Seeded shapes with more than one query head per KV head and chunk
    lengths that are not a multiple of 256, so most are planned on packed
    (token, head) row tiles: GQA ratios 2-8, head_dim 64 and 128, windows that
    wrap the ring, and the split modes auto, none, 5, 16 and balanced."""
    rng = np.random.default_rng(seed)
    shapes = []
    for _ in range(n):
        hkv = int(rng.choice([1, 2]))
        g = int(rng.integers(2, 9))
        d = int(rng.choice([64, 128]))
        c = int(rng.integers(1, 400))
        r = int(rng.integers(64, 1000))
        w = int(rng.integers(0, r + 1))
        shapes.append((ChunkShape(hkv * g, hkv, d, int(rng.integers(0, 80)), r, int(rng.integers(w, 4 * r)), w, c),
                       int(rng.choice([0, 1, 5, 16, -1]))))
    return shapes


RAGGED_GQA = _ragged_gqa_shapes()


def test_ragged_gqa_shapes_are_mostly_packed():
    """(host check of the case list) packing takes fewer row tiles than one
    query head per row tile for most of the cases below"""
    packed = [-(-sh.chunk_len * (sh.num_q_heads // sh.num_kv_heads) // 256) <
              (sh.num_q_heads // sh.num_kv_heads) * -(-sh.chunk_len // 256) for sh, _ in RAGGED_GQA]
    assert sum(packed) >= len(packed) // 2


@pytest.mark.parametrize("case", range(len(RAGGED_GQA)))
@pytest.mark.parametrize("bidir", [False, True])
def test_ragged_gqa_f2_fp32(case, bidir):
    """The seeded ragged GQA shapes, causal and with the bidirectional
    in-chunk option (every row sees the whole chunk)."""
    sh, splits = RAGGED_GQA[case]
    inp = make_chunk_inputs(sh, seed=300 + case, family="F2")
    dc = DeviceChunk(inp)
    flags = vico.VICO_ATTN_BIDIRECTIONAL if bidir else 0
    o, lse = dc.attention(torch.float32, num_splits=splits, flags=flags)
    ref, ref_lse, b = oracle_and_bound(inp, parts=dc.parts, bidirectional=bidir)
    check_f32(o, ref, b, lse, ref_lse)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_f2_bf16(name):
    inp = make_chunk_inputs(SMALL[name], seed=102, family="F2")
    dc = DeviceChunk(inp)
    o, _ = dc.attention(torch.bfloat16)
    ref, _, b = oracle_and_bound(inp, parts=dc.parts)
    check_bf16(o, ref, b)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_f1(name):
    """Literal N(0,1)/sqrt(d) inputs: worst-case and Hoeffding bounds per
    element, relative Frobenius error, LSE."""
    inp = make_chunk_inputs(SMALL[name], seed=103, family="F1")
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.float32)
    ref, ref_lse, b = oracle_and_bound(inp, parts=dc.parts, sigma=True)
    check_f1(o, ref, b)
    check_f32(o, ref, b, lse, ref_lse)


@pytest.mark.parametrize("name", sorted(SMALL))
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_small_f2u_literal_gate(name, out):
    """Outputs bounded by 1: the stated max-abs 1e-2 / mean-abs 1e-3 gate,
    raw and element by element, besides the derived bound."""
    inp = make_chunk_inputs(SMALL[name], seed=104, family="F2U")
    dc = DeviceChunk(inp)
    o, _ = dc.attention(torch.float32 if out == "f32" else torch.bfloat16)
    ref, _, b = oracle_and_bound(inp, parts=dc.parts)
    check_literal(o, ref)
    (check_f32 if out == "f32" else check_bf16)(o, ref, b)


def test_single_visible_key_returns_its_value():
    """Row 0 with no sink and no visible history sees one key: O = V_0 (bf16: exactly)."""
    sh = ChunkShape(4, 2, 128, 0, 64, 300, 0, 33)
    inp = make_chunk_inputs(sh, seed=104, family="F2")
    dc = DeviceChunk(inp)
    ref, _ = oracle_result(inp)
    o16, _ = dc.attention(torch.bfloat16)
    assert np.array_equal(o16[0], ref[0])           # V_0 is bf16, so exact
    o32, _ = dc.attention(torch.float32)
    assert np.max(np.abs(o32[0] - ref[0]) / np.maximum(np.abs(ref[0]), 1e-30)) <= 2.0 ** -21


def _integer_bits(rng, shape, amax):
    """bf16 bits of integers uniform in [-amax, amax] (exact in bf16)."""
    return f32_to_bf16_bits(rng.integers(-amax, amax + 1, shape).astype(np.float32))


def test_large_logits_stay_finite():
    """Integer Q in [-16, 16] and K in [-8, 8]: logits of standard deviation
    ~45 (nats), rows nearly one-hot, so online rescaling is exercised at
    large magnitudes and must not overflow.  Every dot product is an integer
    below 2^24, exact in fp32, so the derived bound is 2^-8 relative to
    sum p|v|/l with almost nothing added."""
    sh = SMALL["gqa7_ragged"]
    inp = make_chunk_inputs(sh, seed=105, family="F2")
    rng = np.random.default_rng(105)
    inp.q = _integer_bits(rng, inp.q.shape, 16)
    for f in ("k_chunk", "sink_k", "hist_k"):
        setattr(inp, f, _integer_bits(rng, getattr(inp, f).shape, 8))
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.float32)
    ref, ref_lse, b = oracle_and_bound(inp, parts=dc.parts, exact_dot=True)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    check_f32(o, ref, b, lse, ref_lse)


@pytest.mark.parametrize("splits", [1, 3, -1])
def test_rising_logits_rescale_often(splits):
    """Keys are small integers times a ramp that rises along the window and
    into the chunk (1 .. 14), so the row maxima keep growing (logit standard
    deviation from ~3 to ~50 nats) and the running max is raised again and
    again: the kernels raise it only when a lane's sum of 16 probabilities
    exceeds 2^8 (or a row has none yet), which happens here both through
    single large probabilities and through many moderately large ones.  Q and
    K are integers, so the logits are exact and the bound is tight."""
    sh = SMALL["gqa7_ragged"]
    inp = make_chunk_inputs(sh, seed=107, family="F2")
    rng = np.random.default_rng(107)
    inp.q = _integer_bits(rng, inp.q.shape, 4)

    def ramp(shape, lo, hi):
        r = np.round(np.linspace(lo, hi, shape[0])).astype(np.float32)[:, None, None]
        return f32_to_bf16_bits(rng.integers(-2, 3, shape).astype(np.float32) * r)
    inp.sink_k = ramp(inp.sink_k.shape, 1, 1)
    inp.hist_k = ramp(inp.hist_k.shape, 1, 10)
    inp.k_chunk = ramp(inp.k_chunk.shape, 10, 14)
    ref, ref_lse, b = oracle_and_bound(inp, exact_dot=True)
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.float32, num_splits=splits)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    b.parts = dc.parts
    check_f32(o, ref, b, lse, ref_lse)
    o16, _ = dc.attention(torch.bfloat16, num_splits=splits)
    check_bf16(o16.astype(np.float64), ref, b)


@pytest.mark.parametrize("scale", [0.05, 0.2, 1.0])
@pytest.mark.parametrize("splits", [1, 3])
def test_explicit_softmax_scale(scale, splits):
    """softmax_scale > 0 replaces 1/sqrt(d).  F2 inputs put the logits' standard
    deviation at ~45 * scale (d = 128): from soft (2.3) to nearly one-hot (45).
    fp32 output and LSE against the oracle at the same scale."""
    inp = make_chunk_inputs(SMALL["gqa7_ragged"], seed=109, family="F2")
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.float32, num_splits=splits, scale=scale)
    ref, ref_lse, b = oracle_and_bound(inp, scale=scale, parts=dc.parts)
    check_f32(o, ref, b, lse, ref_lse)


@pytest.mark.parametrize("splits", [1, 3])
def test_no_lse_and_side_stream_give_the_same_output(splits):
    """The LSE output is optional: without it the output is bit-identical
    (also through the split merge).  The library runs on the caller's stream:
    attention and append issued on a side stream give bit-identical results."""
    inp = make_chunk_inputs(SMALL["gqa7_ragged"], seed=110, family="F2")
    dc = DeviceChunk(inp)
    o_lse, _ = dc.attention(torch.float32, num_splits=splits)
    o_none, l_none = dc.attention(torch.float32, num_splits=splits, with_lse=False)
    assert l_none is None and np.array_equal(o_lse, o_none)

    sh = inp.shape
    ring = [dc.rk.clone(), dc.rv.clone()]
    outs = []
    for stream in (torch.cuda.current_stream(), torch.cuda.Stream()):
        stream.wait_stream(torch.cuda.current_stream())
        rk, rv = ring[0].clone(), ring[1].clone()
        out = torch.empty((sh.chunk_len, sh.num_q_heads, sh.head_dim), dtype=torch.float32, device="cuda")
        _, wb = vico.vico_attn_plan(sh.chunk_len, sh.sink_len, sh.ring_slots, sh.hist_len, sh.window,
                                    sh.num_q_heads, sh.num_kv_heads, sh.head_dim, splits)
        ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
        with torch.cuda.stream(stream):
            vico.vico_chunk_prefill_attn(dc.q, dc.kc, dc.vc, dc.sk, dc.sv, rk, rv, sh.hist_len, sh.window, out,
                                         workspace=ws, num_splits=splits, stream=stream)
            vico.vico_kv_append(dc.kc, dc.vc, rk, rv, sh.hist_len, stream=stream)
        stream.synchronize()
        outs.append((out.clone(), rk, rv))
    assert torch.equal(outs[0][0], outs[1][0])
    assert torch.equal(outs[0][1], outs[1][1]) and torch.equal(outs[0][2], outs[1][2])
    assert np.array_equal(outs[0][0].cpu().numpy().astype(np.float64), o_lse)


def test_split_counts_agree():
    """Every split count meets the derived bound; results differ between split
    counts only by where the bf16 probabilities are rounded (each split keeps
    its own running max), so two of them agree within the sum of their bounds."""
    sh = SMALL["balanced_many_parts"]
    inp = make_chunk_inputs(sh, seed=106, family="F2")
    dc = DeviceChunk(inp)
    x = oracle_and_bound(inp)
    ref, ref_lse, b1 = x
    base, base_lse = dc.attention(torch.float32, num_splits=1)
    check_f32(base, ref, b1, base_lse, ref_lse)
    for ns in (2, 4, 7, 16, -1):
        o, lse = dc.attention(torch.float32, num_splits=ns)
        bn = oracle_and_bound(inp, parts=dc.parts)[2]
        check_f32(o, ref, bn, lse, ref_lse)
        assert np.all(np.abs(o - base) <= bn.f32(ref) + b1.f32(ref))
        assert np.all(np.abs(lse - base_lse) <= bn.lse(ref_lse) + b1.lse(ref_lse))


@pytest.mark.parametrize("cfg", ["7b", "7b_wrap"])
def test_balanced_schedule_agrees_on_every_row(cfg):
    """Full 7B-shaped chunk: the balanced schedule (every work-group an equal
    share of all key tiles; row tiles cut between work-groups and merged by
    log-sum-exp) against the default one, on every row and head, within the
    sum of the two results' derived bounds (sum p|v|/l from the oracle over
    |V| for all rows)."""
    from tests._bounds import chunk_bound
    from tests._util import to_f64
    sh = CONFIGS[cfg]
    inp = make_chunk_inputs(sh, seed=108, family="F2")
    dc = DeviceChunk(inp)
    base, base_lse = dc.attention(torch.float32, num_splits=0)
    p0 = dc.parts
    bal, bal_lse = dc.attention(torch.float32, num_splits=vico.VICO_SPLIT_BALANCED)
    b = chunk_bound(to_f64(inp), parts=max(p0, dc.parts))
    assert np.all(np.isfinite(bal))
    assert np.all(np.abs(bal - base) <= 2.0 * b.f32(base))
    assert np.all(np.abs(bal_lse - base_lse) <= 2.0 * b.lse(base_lse))


def _sample_rows(C, n=40, seed=0):
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(C, size=min(n, C), replace=False).tolist())
    rows |= {0, 1, 31, 32, 127, 128, C - 1}
    return np.array(sorted(r for r in rows if r < C))


FULL = ["3b", "3b_wrap", "7b", "7b_wrap", "full", "full_bounded"]


@pytest.mark.parametrize("cfg", FULL)
def test_full_size_sampled_rows_f2(cfg):
    """Full workload, bf16 output and LSE as benchmarked (auto split), sampled rows vs oracle."""
    sh = CONFIGS[cfg]
    inp = make_chunk_inputs(sh, seed=0, family="F2")
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.bfloat16)
    rows = _sample_rows(sh.chunk_len, seed=1)
    ref, ref_lse, b = oracle_and_bound(inp, rows=rows, parts=dc.parts)
    check_bf16(o[rows], ref, b)
    assert np.all(np.abs(lse[:, rows] - ref_lse) <= b.lse(ref_lse))
    assert np.all(np.isfinite(o))


@pytest.mark.parametrize("cfg", ["3b", "7b_wrap", "full"])
def test_full_size_sampled_rows_f1_fp32(cfg):
    """The benchmarked inputs (N(0,1)/sqrt(d)) at full size: worst-case and
    Hoeffding bounds per element, relative Frobenius error, LSE; the errors
    normalised by rms(O) are what check_f1 returns."""
    sh = CONFIGS[cfg]
    inp = make_chunk_inputs(sh, seed=0, family="F1")
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.float32)
    rows = _sample_rows(sh.chunk_len, seed=2)
    ref, ref_lse, b = oracle_and_bound(inp, rows=rows, parts=dc.parts, sigma=True)
    check_f1(o[rows], ref, b)
    check_f32(o[rows], ref, b, lse[:, rows], ref_lse)


@pytest.mark.parametrize("cfg", ["3b_wrap", "7b_wrap"])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_full_size_sampled_rows_f2u_literal_gate(cfg, out):
    """Full 3B/7B-shaped chunks with outputs bounded by 1 (V uniform in
    [-1, 1]): the stated gate (max-abs 1e-2, mean-abs 1e-3) element by
    element on sampled rows of every row tile, in the launch configuration
    the benchmark times, and the derived bound."""
    sh = CONFIGS[cfg]
    inp = make_chunk_inputs(sh, seed=3, family="F2U")
    dc = DeviceChunk(inp)
    o, _ = dc.attention(torch.float32 if out == "f32" else torch.bfloat16)
    rows = _sample_rows(sh.chunk_len, seed=4)
    ref, _, b = oracle_and_bound(inp, rows=rows, parts=dc.parts)
    check_literal(o[rows], ref)
    (check_f32 if out == "f32" else check_bf16)(o[rows], ref, b)


def _slot_marks(slots):
    """0/1 per ring slot from a multiplicative hash (pattern of the max-size test)."""
    return ((slots * 2654435761) >> 13) & 1


def test_ring_at_the_32bit_offset_limit():
    """Largest ring the kernels address: 2^31 bytes per K/V tensor less one row
    (8388607 slots of one d128 head).  Every key is zero, so every logit is 0:
    a row's output is the plain mean of the V rows it sees and its LSE is
    ln(count), a closed form of the attention definition.  Ring V rows carry a
    slot-hashed 0/1 pattern, so a misaddressed, wrapped-wrong or out-of-range
    read changes the mean.  The window leaves 100000 slots out and wraps at the
    ring end; the slots nearest 2^31 bytes are read.  An append across the
    ring end then lands bit-exact."""
    Hq, Hkv, D, S, C = 2, 1, 128, 16, 64
    R = (1 << 31) // (Hkv * D * 2) - 1
    H = R + 777
    W = R - 100000
    dev = "cuda"
    g = torch.Generator().manual_seed(7)
    cvec = ((torch.arange(D) % 7 - 3) / 4).to(torch.bfloat16)            # exact in bf16
    rk = torch.zeros((R, Hkv, D), dtype=torch.bfloat16, device=dev)
    rv = (_slot_marks(torch.arange(R, device=dev)).to(torch.bfloat16)[:, None] * cvec.to(dev)[None, :])
    rv = rv.reshape(R, Hkv, D)
    sk = torch.zeros((S, Hkv, D), dtype=torch.bfloat16, device=dev)
    sv = torch.randn((S, Hkv, D), generator=g).to(torch.bfloat16)
    kc = torch.zeros((C, Hkv, D), dtype=torch.bfloat16, device=dev)
    vc = torch.randn((C, Hkv, D), generator=g).to(torch.bfloat16)
    q = torch.randn((C, Hq, D), generator=g).to(torch.bfloat16).to(dev)
    ns, wb = vico.vico_attn_plan(C, S, R, H, W, Hq, Hkv, D)
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device=dev)
    out = torch.empty((C, Hq, D), dtype=torch.float32, device=dev)
    lse = torch.empty((Hq, C), dtype=torch.float32, device=dev)
    vico.vico_chunk_prefill_attn(q, kc, vc.to(dev), sk, sv.to(dev), rk, rv, H, W, out, lse=lse, workspace=ws)
    torch.cuda.synchronize()

    # visible ring slots: history tokens H-W .. H-1 live at slots (H-W+k) mod R
    ws0 = (H - W) % R
    vis = np.concatenate([np.arange(ws0, R), np.arange(0, (ws0 + W) - R)]) if ws0 + W > R else np.arange(ws0, ws0 + W)
    assert vis.size == W and ws0 + W > R
    ring_sum = float(_slot_marks(vis.astype(np.int64)).sum()) * cvec.double().numpy()
    sv64, vc64 = sv.double().numpy()[:, 0], vc.double().numpy()[:, 0]
    n = S + W + np.arange(C) + 1
    mean = (sv64.sum(0)[None, :] + ring_sum[None, :] + np.cumsum(vc64, axis=0)) / n[:, None]
    o = out.cpu().double().numpy()
    for h in range(Hq):
        assert np.max(np.abs(o[:, h] - mean)) <= 1e-4
    assert np.max(np.abs(lse.cpu().double().numpy() - np.log(n)[None, :])) <= 1e-4

    # append of 4096 tokens across the ring end
    Ca = 4096
    ka = torch.randn((Ca, Hkv, D), generator=g).to(torch.bfloat16).to(dev)
    va = torch.randn((Ca, Hkv, D), generator=g).to(torch.bfloat16).to(dev)
    p0 = R - 1000
    before = rv[p0 - 1].clone(), rv[Ca - 1000].clone()
    vico.vico_kv_append(ka, va, rk, rv, p0)
    torch.cuda.synchronize()
    assert torch.equal(rk[p0:], ka[:1000]) and torch.equal(rk[:Ca - 1000], ka[1000:])
    assert torch.equal(rv[p0:], va[:1000]) and torch.equal(rv[:Ca - 1000], va[1000:])
    assert torch.equal(rv[p0 - 1], before[0]) and torch.equal(rv[Ca - 1000], before[1])
