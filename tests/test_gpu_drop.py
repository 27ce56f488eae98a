"""GPU parity of temporal token dropping against the oracle (paper, Sec. 3,
"Token Dropping").

The decision is an integer taken on floating-point similarities:
  * the GPU's similarity is within (3 dm + 8) * 2^-24 of the fp64 one (fp32
    sums of dm products; by Cauchy-Schwarz each sum errs by at most dm * 2^-24
    of |x||y|);
  * on its own fp32 similarity the GPU's decision is exact: keep == !(sim > tau);
  * it equals the oracle's wherever the fp64 similarity is further than that
    bound from tau;
  * given its decisions, the retained index list and the copied tokens are
    bit-exact (integer work).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_19849_amd as vico
from synth import DROP_CONFIGS, make_drop_frames
from tests._gpu import bits_of, dev

pytestmark = pytest.mark.gpu
f64 = oracle.bf16_bits_to_f64
U = 2.0 ** -24


def run_gpu(frames_bits, tau, prev_bits=None, with_tokens=True):
    B, C, n_f, dm = frames_bits.shape
    fr = dev(frames_bits)
    keep = torch.full((B, n_f), 7, dtype=torch.uint8, device="cuda")
    sim = torch.full((B, n_f), float("nan"), dtype=torch.float32, device="cuda")
    idx = torch.full((B * C * n_f,), -5, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    out = torch.zeros((B * C * n_f, dm), dtype=torch.bfloat16, device="cuda") if with_tokens else None
    prev = dev(prev_bits) if prev_bits is not None else None
    vico.vico_temporal_drop(fr, tau, keep, idx, cnt, sim=sim, out_tokens=out, prev_frame=prev)
    torch.cuda.synchronize()
    n = int(cnt.item())
    return dict(keep=keep.cpu().numpy(), sim=sim.cpu().numpy(), idx=idx.cpu().numpy(), n=n,
                out=bits_of(out[:n]) if with_tokens else None)


def check(frames_bits, tau, prev_bits=None, with_tokens=True):
    B, C, n_f, dm = frames_bits.shape
    g = run_gpu(frames_bits, tau, prev_bits, with_tokens)
    z = f64(frames_bits)
    keep_ref, sim_ref, _ = oracle.temporal_drop(z, tau, None if prev_bits is None else f64(prev_bits))
    bound = (3 * dm + 8) * U
    assert set(np.unique(g["keep"])) <= {0, 1}
    compared = sim_ref != oracle.NO_COMPARISON
    assert np.all(g["sim"][~compared] == -2.0)
    assert np.max(np.abs(g["sim"][compared] - sim_ref[compared]), initial=0.0) <= bound
    # exact on its own similarity (fp32 comparison with the fp32 threshold)
    assert np.array_equal(g["keep"].astype(bool), ~(g["sim"] > np.float32(tau)))
    clear = np.abs(sim_ref - tau) > bound
    assert np.array_equal(g["keep"].astype(bool)[clear], keep_ref[clear])
    # compaction of the GPU's own decisions: bit-exact
    want = oracle.retained_index(g["keep"].astype(bool), C)
    assert g["n"] == len(want)
    assert np.array_equal(g["idx"][: g["n"]], want)
    if with_tokens:
        assert np.array_equal(g["out"], frames_bits.reshape(B * C * n_f, dm)[want])
    return g, keep_ref


@pytest.mark.parametrize("name", ["tiny", "c2", "c8", "7b", "3b"])
@pytest.mark.parametrize("tau", [0.9, 0.5])
def test_drop_parity(name, tau):
    B, C, n_f, dm = DROP_CONFIGS[name]
    g, keep_ref = check(make_drop_frames(B, C, n_f, dm, seed=B + C + n_f), tau)
    assert 0 < g["keep"].mean() < 1                 # both outcomes occur


@pytest.mark.parametrize("with_prev", [False, True])
def test_frame_level_mode(with_prev):
    B, C, n_f, dm = DROP_CONFIGS["c1"]
    frames = make_drop_frames(B, C, n_f, dm, seed=11)
    prev = make_drop_frames(1, 1, n_f, dm, seed=11)[0, 0] if with_prev else None
    check(frames, 0.8, prev)


def test_indices_only():
    B, C, n_f, dm = DROP_CONFIGS["tiny"]
    check(make_drop_frames(B, C, n_f, dm, seed=12), 0.9, with_tokens=False)


def test_identical_frames_keep_only_anchors():
    base = make_drop_frames(3, 1, 40, 128, seed=13)
    frames = np.repeat(base, 4, axis=1)
    g, _ = check(frames, 0.5)
    assert not g["keep"].any() and g["n"] == 3 * 40


def test_exact_cosine_at_the_threshold_is_kept():
    """(3, 4) and (4, 3) have cosine 24/25: exact in fp32 (norms 5, dot 24),
    so tau = 0.96 (as fp32) must not drop, and any smaller tau must."""
    frames = np.zeros((1, 2, 4, 64), dtype=np.float32)
    frames[0, 0, :, :2] = (3, 4)
    frames[0, 1, :, :2] = (4, 3)
    bits = frames.view(np.uint32).__rshift__(16).astype(np.uint16)       # exact: small integers
    g = run_gpu(bits, float(np.float32(0.96)))
    assert np.all(g["sim"] == np.float32(0.96)) and g["keep"].all()
    g = run_gpu(bits, float(np.nextafter(np.float32(0.96), np.float32(0))))
    assert not g["keep"].any()


def test_zero_vectors_score_zero():
    frames = np.zeros((2, 3, 8, 32), dtype=np.uint16)
    frames[:, :, 4:, 0] = 0x3F80                                        # 1.0 at the last four positions
    g = run_gpu(frames, -0.5)
    assert np.all(g["sim"][:, :4] == 0) and np.all(g["sim"][:, 4:] == 1) and not g["keep"].any()


def test_many_chunks_ranks_across_chunks():
    """64 chunks of the 3B shape at tau 0.9: output offsets of each chunk depend
    on the counts of all earlier chunks."""
    frames = make_drop_frames(64, 4, 64, 256, seed=14)
    check(frames, 0.9)
