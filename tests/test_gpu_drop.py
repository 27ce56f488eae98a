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


SCHEDULES = ["two_pass", "single_pass"]


def workspace_for(shape, schedule, fill=0xFF):
    """The workspace that selects `schedule` (None: two passes); filled with
    garbage, since the call must not rely on its contents."""
    if schedule == "two_pass":
        return None
    nb = vico.vico_temporal_drop_workspace_bytes(*shape)
    assert nb > 0, f"{shape}: the single pass should apply"
    return torch.full((nb,), fill, dtype=torch.uint8, device="cuda")


def run_gpu(frames_bits, tau, prev_bits=None, with_tokens=True, schedule="two_pass", workspace=None):
    B, C, n_f, dm = frames_bits.shape
    if workspace is None:
        workspace = workspace_for(frames_bits.shape, schedule)
    fr = dev(frames_bits)
    keep = torch.full((B, n_f), 7, dtype=torch.uint8, device="cuda")
    sim = torch.full((B, n_f), float("nan"), dtype=torch.float32, device="cuda")
    idx = torch.full((B * C * n_f,), -5, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    out = torch.zeros((B * C * n_f, dm), dtype=torch.bfloat16, device="cuda") if with_tokens else None
    prev = dev(prev_bits) if prev_bits is not None else None
    vico.vico_temporal_drop(fr, tau, keep, idx, cnt, sim=sim, out_tokens=out, prev_frame=prev, workspace=workspace)
    torch.cuda.synchronize()
    n = int(cnt.item())
    return dict(keep=keep.cpu().numpy(), sim=sim.cpu().numpy(), idx=idx.cpu().numpy(), n=n,
                out=bits_of(out[:n]) if with_tokens else None)


def check(frames_bits, tau, prev_bits=None, with_tokens=True, schedule="two_pass"):
    B, C, n_f, dm = frames_bits.shape
    g = run_gpu(frames_bits, tau, prev_bits, with_tokens, schedule)
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


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("name", ["tiny", "c2", "c8", "7b", "3b"])
@pytest.mark.parametrize("tau", [0.9, 0.5])
def test_drop_parity(name, tau, schedule):
    B, C, n_f, dm = DROP_CONFIGS[name]
    g, keep_ref = check(make_drop_frames(B, C, n_f, dm, seed=B + C + n_f), tau, schedule=schedule)
    assert 0 < g["keep"].mean() < 1                 # both outcomes occur


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("with_prev", [False, True])
def test_frame_level_mode(with_prev, schedule):
    B, C, n_f, dm = DROP_CONFIGS["c1"]
    frames = make_drop_frames(B, C, n_f, dm, seed=11)
    prev = make_drop_frames(1, 1, n_f, dm, seed=11)[0, 0] if with_prev else None
    check(frames, 0.8, prev, schedule=schedule)


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_indices_only(schedule):
    B, C, n_f, dm = DROP_CONFIGS["tiny"]
    check(make_drop_frames(B, C, n_f, dm, seed=12), 0.9, with_tokens=False, schedule=schedule)


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_identical_frames_keep_only_anchors(schedule):
    base = make_drop_frames(3, 1, 40, 128, seed=13)
    frames = np.repeat(base, 4, axis=1)
    g, _ = check(frames, 0.5, schedule=schedule)
    assert not g["keep"].any() and g["n"] == 3 * 40


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_exact_cosine_at_the_threshold_is_kept(schedule):
    """(3, 4) and (4, 3) have cosine 24/25: exact in fp32 (norms 5, dot 24),
    so tau = 0.96 (as fp32) must not drop, and any smaller tau must."""
    frames = np.zeros((1, 2, 4, 64), dtype=np.float32)
    frames[0, 0, :, :2] = (3, 4)
    frames[0, 1, :, :2] = (4, 3)
    bits = frames.view(np.uint32).__rshift__(16).astype(np.uint16)       # exact: small integers
    g = run_gpu(bits, float(np.float32(0.96)), schedule=schedule)
    assert np.all(g["sim"] == np.float32(0.96)) and g["keep"].all()
    g = run_gpu(bits, float(np.nextafter(np.float32(0.96), np.float32(0))), schedule=schedule)
    assert not g["keep"].any()


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_zero_vectors_score_zero(schedule):
    frames = np.zeros((2, 3, 8, 32), dtype=np.uint16)
    frames[:, :, 4:, 0] = 0x3F80                                        # 1.0 at the last four positions
    g = run_gpu(frames, -0.5, schedule=schedule)
    assert np.all(g["sim"][:, :4] == 0) and np.all(g["sim"][:, 4:] == 1) and not g["keep"].any()


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_many_chunks_ranks_across_chunks(schedule):
    """64 chunks of the 3B shape at tau 0.9: output offsets of each chunk depend
    on the counts of all earlier chunks."""
    frames = make_drop_frames(64, 4, 64, 256, seed=14)
    check(frames, 0.9, schedule=schedule)


@pytest.mark.parametrize("shape,tau,with_prev", [
    ((150, 2, 40, 128), 0.9, False),     # the look-back spans three windows of 64 chunks
    ((5, 1, 1024, 64), 0.8, True),       # 256 tiles per chunk, the most the single pass takes
    ((7, 3, 37, 4096), 0.9, False),      # 8 units of 512 features per lane, ragged tiles
    ((4, 8, 50, 2048), 0.5, False),      # C = 8 at its widest single-pass row
    ((9, 1, 13, 200), 0.8, False),       # C = 1 without a previous frame; 25 pieces of a row
    ((9, 3, 1, 64), 0.5, False),         # one position per frame: every group leads its chunk
    ((7, 4, 3, 128), 0.5, False),        # one ragged tile per chunk
    ((256, 2, 4, 64), 0.9, False),       # the most chunks the single pass takes: a look-back of 4 windows
    ((6, 4, 37, 8), 0.5, False),         # 8 features: one lane of a wave holds the row
])
def test_schedules_agree_bit_for_bit(shape, tau, with_prev):
    """Both schedules run the same arithmetic: every output is the same bits,
    and the single pass meets the oracle on its own."""
    B, C, n_f, dm = shape
    frames = make_drop_frames(B, C, n_f, dm, seed=B * 31 + C)
    prev = make_drop_frames(1, 1, n_f, dm, seed=B * 31 + C + 1)[0, 0] if with_prev else None
    one, _ = check(frames, tau, prev, schedule="single_pass")
    two = run_gpu(frames, tau, prev, schedule="two_pass")
    assert one["n"] == two["n"]
    for k in ("keep", "idx", "out"):
        assert np.array_equal(one[k], two[k]), k
    assert np.array_equal(one["sim"].view(np.uint32), two["sim"].view(np.uint32))


@pytest.mark.parametrize("shape,tau,with_prev", [
    ((5, 4, 24, 256), 0.9, False),
    ((4, 1, 13, 200), 0.8, True),
    ((3, 1, 9, 64), 0.8, False),
    ((70, 2, 8, 64), 0.9, False),        # chunk counts beyond one window of 64
])
def test_single_pass_recount_path(monkeypatch, shape, tau, with_prev):
    """With no time to wait, every group recounts what it needs from the
    frames: the results are still those of the two passes, bit for bit."""
    B, C, n_f, dm = shape
    frames = make_drop_frames(B, C, n_f, dm, seed=B * 7 + C)
    prev = make_drop_frames(1, 1, n_f, dm, seed=B * 7 + C + 1)[0, 0] if with_prev else None
    two = run_gpu(frames, tau, prev, schedule="two_pass")
    monkeypatch.setenv("VICO_DROP_WAIT_US", "0")
    one = run_gpu(frames, tau, prev, schedule="single_pass")
    assert one["n"] == two["n"]
    for k in ("keep", "idx", "out"):
        assert np.array_equal(one[k], two[k]), k
    assert np.array_equal(one["sim"].view(np.uint32), two["sim"].view(np.uint32))


def test_single_pass_workspace_reuse():
    """One workspace across calls of different sizes, on one stream: each call
    starts from its own zeroed control block."""
    big = make_drop_frames(16, 4, 96, 512, seed=21)
    small = make_drop_frames(3, 4, 40, 512, seed=22)
    ws = workspace_for(big.shape, "single_pass")
    for frames in (big, small, big):
        one = run_gpu(frames, 0.9, schedule="single_pass", workspace=ws)
        two = run_gpu(frames, 0.9, schedule="two_pass")
        assert one["n"] == two["n"] and one["n"] > 0
        for k in ("keep", "idx", "out"):
            assert np.array_equal(one[k], two[k]), k


def test_single_pass_not_covered_runs_two_passes():
    """A workspace with a shape the single pass does not take is ignored."""
    B, C, n_f, dm = 2, 8, 24, 2056
    assert vico.vico_temporal_drop_workspace_bytes(B, C, n_f, dm) == 0
    ws = torch.full((256,), 0xFF, dtype=torch.uint8, device="cuda")
    frames = make_drop_frames(B, C, n_f, dm, seed=23)
    two, _ = check(frames, 0.5, schedule="two_pass")
    given = run_gpu(frames, 0.5, workspace=ws)
    assert given["n"] == two["n"]
    for k in ("keep", "idx", "out"):
        assert np.array_equal(given[k], two[k]), k
    assert torch.all(ws == 0xFF)                     # untouched


def test_drop_with_workspace_replays_as_a_graph():
    """Captured into a HIP graph, a call with a workspace takes the two passes
    (the single pass tags its words per call, which replays would repeat): the
    replays reproduce the eager result, with eager single-pass calls on other
    inputs and the same buffers in between."""
    B, C, n_f, dm = 6, 4, 40, 512
    frames = [dev(make_drop_frames(B, C, n_f, dm, seed=31 + i)) for i in range(2)]
    ws = workspace_for((B, C, n_f, dm), "single_pass")
    keep = torch.empty((B, n_f), dtype=torch.uint8, device="cuda")
    idx = torch.empty(B * C * n_f, dtype=torch.int32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    out = torch.empty((B * C * n_f, dm), dtype=torch.bfloat16, device="cuda")

    def step(i):
        vico.vico_temporal_drop(frames[i], 0.9, keep, idx, cnt, out_tokens=out, workspace=ws)

    eager = []
    for i in range(2):
        step(i)
        torch.cuda.synchronize()
        n = int(cnt.item())
        eager.append((keep.clone(), idx[:n].clone(), out[:n].clone(), n))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        step(0)
        torch.cuda.current_stream().synchronize()
        with torch.cuda.graph(graph, stream=side):
            step(0)
    torch.cuda.synchronize()
    for _ in range(3):
        step(1)
        torch.cuda.synchronize()
        k, i1, o, n = eager[1]
        assert int(cnt.item()) == n and torch.equal(keep, k) and torch.equal(idx[:n], i1) and torch.equal(out[:n], o)
        keep.fill_(7)
        idx.fill_(-5)
        graph.replay()
        torch.cuda.synchronize()
        k, i0, o, n = eager[0]
        assert int(cnt.item()) == n and torch.equal(keep, k) and torch.equal(idx[:n], i0) and torch.equal(out[:n], o)


def test_single_pass_back_to_back_and_concurrent_calls():
    """Calls queued back to back on one stream with one workspace, and calls on
    two streams at once with their own workspaces: every call's words carry
    its own tag, so each result is that of the two passes on its inputs."""
    shapes = [(12, 4, 64, 512), (5, 4, 40, 512), (12, 4, 64, 512)]
    frames = [make_drop_frames(*s, seed=41 + i) for i, s in enumerate(shapes)]
    want = [run_gpu(f, 0.9, schedule="two_pass") for f in frames]

    def prepare(bits):
        B, C, n_f, dm = bits.shape
        return dict(fr=dev(bits), keep=torch.full((B, n_f), 7, dtype=torch.uint8, device="cuda"),
                    idx=torch.full((B * C * n_f,), -5, dtype=torch.int32, device="cuda"),
                    cnt=torch.full((1,), -1, dtype=torch.int32, device="cuda"),
                    out=torch.zeros((B * C * n_f, dm), dtype=torch.bfloat16, device="cuda"))

    def launch(o, ws, stream):
        with torch.cuda.stream(stream):
            vico.vico_temporal_drop(o["fr"], 0.9, o["keep"], o["idx"], o["cnt"], out_tokens=o["out"], workspace=ws,
                                    stream=stream)

    def same(o, w):
        n = int(o["cnt"].item())
        assert n == w["n"]
        assert np.array_equal(o["keep"].cpu().numpy(), w["keep"])
        assert np.array_equal(o["idx"].cpu().numpy()[:n], w["idx"][:n])
        assert np.array_equal(bits_of(o["out"][:n]), w["out"])

    ws, ws2 = workspace_for(shapes[0], "single_pass"), workspace_for(shapes[0], "single_pass")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = [prepare(f) for f in frames]
    torch.cuda.synchronize()
    for o in outs:
        launch(o, ws, s1)                                 # queued on s1, no wait between
    torch.cuda.synchronize()
    for o, w in zip(outs, want):
        same(o, w)
    o1, o2 = prepare(frames[0]), prepare(frames[2])
    torch.cuda.synchronize()
    launch(o1, ws, s1)
    launch(o2, ws2, s2)
    torch.cuda.synchronize()
    same(o1, want[0])
    same(o2, want[2])
