"""GPU parity: the HIP attention path against the fp64 oracle, element by element.

Small shapes are compared in full; the full-size workloads (3B/7B layer
shapes, full-history 65536 tokens) run the whole chunk on the GPU in the
launch configuration the benchmark times and are compared on sampled rows.

Tolerances
  * F2 inputs (Q, K ~ 2 N(0,1); V ~ N(0,1): logits of std 4, O(1) outputs),
    fp32 output: max-abs <= 1e-2 per unit of output magnitude (bf16 P rounding
    is relative) and mean-abs <= 1e-3;
    LSE max-abs <= 1e-3.
  * bf16 output: the same plus half a bf16 ulp of output rounding.
  * F1 inputs (N(0,1)/sqrt(d), outputs ~1e-3): relative Frobenius error
    <= 5e-3, since an absolute bound would pass a zero output.
"""
import numpy as np
import pytest
import torch

from oracle import bf16_bits_to_f64
from synth import CONFIGS, ChunkShape, f32_to_bf16_bits, make_chunk_inputs
from tests._gpu import DeviceChunk, check_bf16, check_f32, check_relative, oracle_result

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
    o, lse = DeviceChunk(inp).attention(torch.float32, num_splits=splits)
    ref, ref_lse = oracle_result(inp)
    check_f32(o, ref, lse, ref_lse)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_f2_bf16(name):
    inp = make_chunk_inputs(SMALL[name], seed=102, family="F2")
    o, _ = DeviceChunk(inp).attention(torch.bfloat16)
    ref, _ = oracle_result(inp)
    check_bf16(o, ref)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_f1_relative(name):
    inp = make_chunk_inputs(SMALL[name], seed=103, family="F1")
    o, lse = DeviceChunk(inp).attention(torch.float32)
    ref, ref_lse = oracle_result(inp)
    check_relative(o, ref)
    assert np.max(np.abs(lse - ref_lse)) <= 1e-3


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


def test_large_logits_stay_finite():
    """Q scaled x50 on F2 inputs (logit std ~200): online rescaling must not overflow.
    Rows are then nearly one-hot, so the bf16 rounding of the largest
    probabilities (2^-9 relative) shows up almost undiluted: max-abs 5e-2."""
    sh = SMALL["gqa7_ragged"]
    inp = make_chunk_inputs(sh, seed=105, family="F2")
    inp.q = f32_to_bf16_bits(bf16_bits_to_f64(inp.q).astype(np.float32) * 50)
    o, lse = DeviceChunk(inp).attention(torch.float32)
    ref, ref_lse = oracle_result(inp)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    check_f32(o, ref, lse, ref_lse, max_abs=5e-2, mean_abs=2e-3, lse_abs=1e-3)


@pytest.mark.parametrize("splits", [1, 3, -1])
def test_rising_logits_rescale_often(splits):
    """Keys scaled by a ramp that rises along the window and into the chunk, so
    the row maxima keep growing and the running max is raised again and again:
    the kernels raise it only when a lane's sum of 16 probabilities exceeds
    2^8 (or a row has none yet), which happens here both through single large
    probabilities and through many moderately large ones.  Peaked rows, so the
    bound of the large-logit test applies."""
    sh = SMALL["gqa7_ragged"]
    inp = make_chunk_inputs(sh, seed=107, family="F2")
    def ramp(bits, lo, hi):
        x = bf16_bits_to_f64(bits).astype(np.float32)
        r = np.linspace(lo, hi, x.shape[0], dtype=np.float32)[:, None, None]
        return f32_to_bf16_bits(x * r)
    inp.hist_k = ramp(inp.hist_k, 0.25, 2.5)
    inp.k_chunk = ramp(inp.k_chunk, 2.5, 3.5)
    ref, ref_lse = oracle_result(inp)
    dc = DeviceChunk(inp)
    o, lse = dc.attention(torch.float32, num_splits=splits)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    check_f32(o, ref, lse, ref_lse, max_abs=5e-2, mean_abs=2e-3, lse_abs=1e-3)
    o16, _ = dc.attention(torch.bfloat16, num_splits=splits)
    assert np.max(np.abs(o16.astype(np.float64) - o)) <= 2e-2 * max(1.0, float(np.max(np.abs(o))))


@pytest.mark.parametrize("scale", [0.05, 0.2, 1.0])
@pytest.mark.parametrize("splits", [1, 3])
def test_explicit_softmax_scale(scale, splits):
    """softmax_scale > 0 replaces 1/sqrt(d).  F2 inputs put the logits' standard
    deviation at ~45 * scale (d = 128): from soft (2.3) to nearly one-hot (45).
    fp32 output and LSE against the oracle at the same scale."""
    inp = make_chunk_inputs(SMALL["gqa7_ragged"], seed=109, family="F2")
    o, lse = DeviceChunk(inp).attention(torch.float32, num_splits=splits, scale=scale)
    ref, ref_lse = oracle_result(inp, scale=scale)
    check_f32(o, ref, lse, ref_lse)


@pytest.mark.parametrize("splits", [1, 3])
def test_no_lse_and_side_stream_give_the_same_output(splits):
    """The LSE output is optional: without it the output is bit-identical
    (also through the split merge).  The library runs on the caller's stream:
    attention and append issued on a side stream give bit-identical results."""
    import paper_2606_19849_amd as vico
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
    """Every split count meets the oracle tolerance; results differ between split
    counts only by where the bf16 probabilities are rounded (each split keeps its
    own running max), so two of them agree within twice the per-result bound."""
    sh = SMALL["balanced_many_parts"]
    inp = make_chunk_inputs(sh, seed=106, family="F2")
    dc = DeviceChunk(inp)
    ref, ref_lse = oracle_result(inp)
    base, base_lse = dc.attention(torch.float32, num_splits=1)
    check_f32(base, ref, base_lse, ref_lse)
    for ns in (2, 4, 7, 16, -1):
        o, lse = dc.attention(torch.float32, num_splits=ns)
        check_f32(o, ref, lse, ref_lse)
        assert np.max(np.abs(o - base)) <= 2e-2
        assert np.max(np.abs(lse - base_lse)) <= 2e-3


@pytest.mark.parametrize("cfg", ["7b", "7b_wrap"])
def test_balanced_schedule_agrees_on_every_row(cfg):
    """Full 7B-shaped chunk: the balanced schedule (every work-group an equal
    share of all key tiles; row tiles cut between work-groups and merged by
    log-sum-exp) against the default one, on every row and head."""
    import paper_2606_19849_amd as vico
    sh = CONFIGS[cfg]
    inp = make_chunk_inputs(sh, seed=108, family="F2")
    dc = DeviceChunk(inp)
    base, base_lse = dc.attention(torch.float32, num_splits=0)
    bal, bal_lse = dc.attention(torch.float32, num_splits=vico.VICO_SPLIT_BALANCED)
    assert np.all(np.isfinite(bal))
    assert np.max(np.abs(bal - base)) <= 2e-2
    assert np.mean(np.abs(bal - base)) <= 1e-3
    assert np.max(np.abs(bal_lse - base_lse)) <= 2e-3


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
    o, lse = DeviceChunk(inp).attention(torch.bfloat16)
    rows = _sample_rows(sh.chunk_len, seed=1)
    ref, ref_lse = oracle_result(inp, rows=rows)
    check_bf16(o[rows], ref)
    assert np.max(np.abs(lse[:, rows] - ref_lse)) <= 1e-3
    assert np.all(np.isfinite(o))


@pytest.mark.parametrize("cfg", ["3b", "7b_wrap", "full"])
def test_full_size_sampled_rows_f1_fp32(cfg):
    sh = CONFIGS[cfg]
    inp = make_chunk_inputs(sh, seed=0, family="F1")
    o, lse = DeviceChunk(inp).attention(torch.float32)
    rows = _sample_rows(sh.chunk_len, seed=2)
    ref, ref_lse = oracle_result(inp, rows=rows)
    check_relative(o[rows], ref)
    assert np.max(np.abs(lse[:, rows] - ref_lse)) <= 1e-3


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
    import paper_2606_19849_amd as vico
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
