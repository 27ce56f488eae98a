"""Host-side checks of the C ABI: the library loads, exports every function the
header declares, plans launches, and rejects bad arguments before any HIP call.
None of these tests touches a GPU."""
import ctypes

import pytest

import paper_2606_19849_amd as vico
from synth import CONFIGS

lib = vico.load_library()
A = 0x10000          # fake, 16-byte aligned "device" addresses: validation never dereferences them
B = 0x20000000
MIS = 0x10008

EXPECTED = {"vico_kv_append", "vico_chunk_prefill_attn", "vico_attn_plan", "vico_attn_workspace_bytes",
            "vico_status_str", "vico_last_hip_error", "vico_token_mean", "vico_chunk_scores", "vico_topk_chunks",
            "vico_gather_plan", "vico_gather_attn", "vico_chunk_prefill_attn_ex", "vico_attn_plan_ex",
            "vico_acn_window", "vico_temporal_drop", "vico_gather_attn_noalloc",
            "vico_temporal_drop_workspace_bytes"}


def test_header_declares_the_expected_entry_points():
    assert set(vico.header_functions()) == EXPECTED


@pytest.mark.parametrize("name", sorted(EXPECTED))
def test_library_exports_every_header_symbol(name):
    assert hasattr(lib, name)


def test_single_hip_runtime_in_process():
    """libvico resolves libamdhip64 to the copy torch already loaded."""
    paths = set()
    for line in open("/proc/self/maps"):
        if "libamdhip64" in line:
            paths.add(line.split()[-1])
    assert len(paths) == 1, paths


def test_status_strings():
    for s in range(-7, 1):
        assert lib.vico_status_str(s) and lib.vico_status_str(s) != b"unknown status"
    assert lib.vico_status_str(-99) == b"unknown status"
    assert lib.vico_last_hip_error() == 0


def _attn(**kw):
    a = dict(q=A, kc=A + 0x100000, vc=A + 0x200000, C=64, sk=A + 0x300000, sv=A + 0x400000, S=16,
             rk=A + 0x500000, rv=A + 0x600000, R=256, H=456, W=256, Hq=2, Hkv=1, D=64, scale=0.0,
             out=B, odt=1, lse=None, splits=0, ws=None, wsb=0, stream=None)
    a.update(kw)
    return lib.vico_chunk_prefill_attn(a["q"], a["kc"], a["vc"], a["C"], a["sk"], a["sv"], a["S"], a["rk"],
                                       a["rv"], a["R"], a["H"], a["W"], a["Hq"], a["Hkv"], a["D"], a["scale"],
                                       a["out"], a["odt"], a["lse"], a["splits"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(Hq=3, Hkv=2), -1),                 # heads not grouped evenly
    (dict(Hkv=0), -1),
    (dict(D=96), -2),                        # unsupported head_dim
    (dict(W=-2), -1),
    (dict(C=-1), -1),
    (dict(S=-1), -1),
    (dict(H=-5), -1),
    (dict(R=128), -3),                       # window 256 does not fit a 128-slot ring
    (dict(W=-1, H=300), -3),                 # full history already partly evicted
    (dict(q=None), -1),
    (dict(out=None), -1),
    (dict(sk=None), -1),                     # sink pointers required when S > 0
    (dict(rk=None), -1),                     # ring pointers required when Wv > 0
    (dict(q=MIS), -4),
    (dict(out=B + 4), -4),
    (dict(lse=B + 0x100002), -4),
    (dict(odt=7), -2),
    (dict(scale=float("nan")), -1),
    (dict(splits=-2), -1),
    (dict(out=A + 8 * 16), -1),              # output aliases q
    (dict(lse=A + 0x500000 + 64), -1),       # lse aliases the ring
    (dict(C=1 << 21), -1),                   # chunk beyond the supported maximum
])
def test_attention_rejects_bad_arguments(kw, status):
    assert _attn(**kw) == status


def test_attention_accepts_null_ring_when_no_history_is_visible():
    # window 0 and no sink: nothing to validate on the ring side; C == 0 returns before launching
    assert _attn(C=0, rk=None, rv=None, W=0, S=0, sk=None, sv=None) == 0


def test_empty_chunk_is_a_noop():
    assert _attn(C=0, q=None, kc=None, vc=None, out=None) == 0
    assert lib.vico_kv_append(None, None, 0, None, None, 16, 5, 1, 64, None) == 0


def test_split_workspace_is_required():
    # 3B shape plans 4 splits and needs a workspace
    sh = CONFIGS["3b"]
    ns, wb = vico.vico_attn_plan(sh.chunk_len, sh.sink_len, sh.ring_slots, sh.hist_len, sh.window,
                                 sh.num_q_heads, sh.num_kv_heads, sh.head_dim)
    assert ns > 1 and wb > 0
    assert _attn(C=sh.chunk_len, S=sh.sink_len, R=sh.ring_slots, H=sh.hist_len, W=sh.window, Hq=16, Hkv=2,
                 D=128, q=A, kc=A + (1 << 26), vc=A + (2 << 26), sk=A + (3 << 26), sv=A + (4 << 26),
                 rk=A + (5 << 26), rv=A + (6 << 26), out=B, ws=None, wsb=0) == -5
    assert _attn(C=sh.chunk_len, S=sh.sink_len, R=sh.ring_slots, H=sh.hist_len, W=sh.window, Hq=16, Hkv=2,
                 D=128, q=A, kc=A + (1 << 26), vc=A + (2 << 26), sk=A + (3 << 26), sv=A + (4 << 26),
                 rk=A + (5 << 26), rv=A + (6 << 26), out=B, ws=B + (1 << 30), wsb=wb - 1) == -5


# 7B: 28 heads x 8 row tiles of 256 rows = 224 work-groups for 256 CUs: no merge
@pytest.mark.parametrize("cfg,splits", [("tiny", {1}), ("tiny_partial", {1}), ("3b", {4}), ("3b_wrap", {4}),
                                        ("7b", {1}), ("7b_wrap", {1}), ("full", {2}), ("full_bounded", {2})])
def test_plan_for_the_workloads(cfg, splits):
    sh = CONFIGS[cfg]
    ns, wb = vico.vico_attn_plan(sh.chunk_len, sh.sink_len, sh.ring_slots, sh.hist_len, sh.window,
                                 sh.num_q_heads, sh.num_kv_heads, sh.head_dim)
    assert ns in splits
    if ns == 1:
        assert wb == 0
    else:
        C, Hq, D = sh.chunk_len, sh.num_q_heads, sh.head_dim
        o_bytes = (4 * ns * Hq * C * D + 255) // 256 * 256
        assert wb == o_bytes + 4 * ns * Hq * C
    assert vico.vico_attn_workspace_bytes(sh.chunk_len, sh.sink_len, sh.ring_slots, sh.hist_len, sh.window,
                                          sh.num_q_heads, sh.num_kv_heads, sh.head_dim) == wb


# 3B heads (16q/2kv) with a full 8192-token window, the 64-chunk stream's
# shapes: a chunk length that is not a multiple of 256 is planned on packed
# (token, head) row tiles, ceil(C * 8 / 256) per KV head, which leaves room for
# more key splits in one round of 256 work-groups (at most 16, and at least 8
# key tiles per split); whole 256-row tiles stay one query head per tile
@pytest.mark.parametrize("C,splits", [(258, 14), (300, 12), (390, 9), (512, 8), (640, 6), (700, 5), (800, 5),
                                      (1000, 4), (1024, 4)])
def test_plan_for_ragged_stream_chunks(C, splits):
    ns, wb = vico.vico_attn_plan(C, 64, 8192, 5 * 8192 + 777, 8192, 16, 2, 128)
    assert ns == splits
    assert wb == (4 * ns * 16 * C * 128 + 255) // 256 * 256 + 4 * ns * 16 * C


def test_forced_splits_are_clamped_to_the_key_tiles():
    # 16 + 256 + 64 keys in tiles of 64 keys -> at most 6 splits
    assert vico.vico_attn_plan(64, 16, 256, 456, 256, 2, 1, 64, num_splits=8)[0] == 6
    assert vico.vico_attn_plan(64, 16, 256, 456, 256, 2, 1, 64, num_splits=2)[0] == 2
    # and to 16 (the row merge loads up to 16 parts at once)
    assert vico.vico_attn_plan(64, 16, 4096, 5000, 4096, 2, 1, 64, num_splits=40)[0] == 16
    with pytest.raises(vico.VicoError):
        vico.vico_attn_plan(64, 16, 256, 456, 256, 2, 1, 64, num_splits=-3)


def test_balanced_plan_needs_enough_key_tiles():
    # 6 key tiles in total cannot be shared by 256 work-groups: fall back to one per row tile
    assert vico.vico_attn_plan(64, 16, 256, 456, 256, 2, 1, 64, num_splits=vico.VICO_SPLIT_BALANCED)[0] == 1
    # 7B shape: partials per row are bounded and the workspace holds them
    ns, wb = vico.vico_attn_plan(2048, 64, 16384, 16384, 16384, 28, 4, 128, num_splits=vico.VICO_SPLIT_BALANCED)
    assert 2 <= ns <= 3 and wb == (4 * ns * 28 * 2048 * 128 + 255) // 256 * 256 + 4 * ns * 28 * 2048


@pytest.mark.parametrize("args,status", [
    ((A, A + 0x1000, 17, B, B + 0x100000, 16, 0, 1, 64), -3),     # chunk longer than the ring
    ((A, A + 0x1000, 4, B, B + 0x100000, 16, -1, 1, 64), -1),
    ((A, A + 0x1000, 4, B, B + 0x100000, 16, 0, 1, 80), -2),
    ((A, A + 0x1000, 4, B, B + 0x100000, 16, 0, 0, 64), -1),
    ((MIS, A + 0x1000, 4, B, B + 0x100000, 16, 0, 1, 64), -4),
    ((A, A + 0x1000, 4, None, B + 0x100000, 16, 0, 1, 64), -1),
    ((A, A + 0x1000, 4, B, B + 64, 16, 0, 1, 64), -1),             # ring_k and ring_v overlap
    ((B + 128, A + 0x1000, 4, B, B + 0x100000, 16, 0, 1, 64), -1),  # chunk inside the ring
])
def test_append_rejects_bad_arguments(args, status):
    assert lib.vico_kv_append(*args, None) == status


# ---------------------------------------------------------------- retrieval entry points

@pytest.mark.parametrize("args,status", [
    ((A, 0, 64, B), -1),                     # no tokens
    ((A, 8, 60, B), -1),                     # feat_dim not a multiple of 8
    ((None, 8, 64, B), -1),
    ((A, 8, 64, None), -1),
    ((MIS, 8, 64, B), -4),
    ((A, 8, 64, B + 4), -4),
    ((A, 8, 64, A + 16), -1),                # out inside x
])
def test_token_mean_rejects_bad_arguments(args, status):
    assert lib.vico_token_mean(*args, None) == status


@pytest.mark.parametrize("args,status", [
    ((A, B, -1, 64, B + 0x100000), -1),
    ((A, B, 4, 12, B + 0x100000), -1),
    ((None, B, 4, 64, B + 0x100000), -1),
    ((A, B, 4, 64, None), -1),
    ((MIS, B, 4, 64, B + 0x100000), -4),
    ((A, B, 4, 64, B + 0x100), -1),          # scores inside the feature table
])
def test_chunk_scores_rejects_bad_arguments(args, status):
    assert lib.vico_chunk_scores(*args, None) == status


def test_chunk_scores_of_no_chunks_is_a_no_op():
    assert lib.vico_chunk_scores(A, B, 0, 64, None, None) == 0


def _topk(**kw):
    a = dict(sc=A, N=100, k=8, tau=float("-inf"), cs=A + 0x1000, cl=A + 0x2000, oc=B, os=B + 0x100,
             ss=B + 0x200, sl=B + 0x300, cnt=B + 0x400)
    a.update(kw)
    return lib.vico_topk_chunks(a["sc"], a["N"], a["k"], a["tau"], a["cs"], a["cl"], a["oc"], a["os"], a["ss"],
                                a["sl"], a["cnt"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(k=0), -1),
    (dict(k=2049), -1),
    (dict(N=-1), -1),
    (dict(tau=float("nan")), -1),
    (dict(sc=None), -1),
    (dict(oc=None), -1),
    (dict(cnt=None), -1),
    (dict(cl=None), -1),                     # chunk table given by halves
    (dict(ss=None), -1),                     # chunk table without a segment output
    (dict(cs=A + 0x1004), -4),               # int64 table not 8-byte aligned
    (dict(oc=B + 2), -4),
    (dict(os=B + 0x10), -1),                 # out_scores overlaps out_chunks
    (dict(oc=A + 0x40), -1),                 # output inside the scores
])
def test_topk_rejects_bad_arguments(kw, status):
    assert _topk(**kw) == status


def _gather(**kw):
    a = dict(q=A, Lq=4, tk=A + 0x100000, tv=A + 0x200000, T=6, sk=A + 0x300000, sv=A + 0x400000, S=8,
             gk=A + 0x500000, gv=A + 0x600000, cap=500, ss=A + 0x700000, sl=A + 0x701000, n=3, hint=100,
             Hq=2, Hkv=1, D=64, scale=0.0, out=B, odt=1, lse=None, splits=0, ws=None, wsb=0)
    a.update(kw)
    return lib.vico_gather_attn(a["q"], a["Lq"], a["tk"], a["tv"], a["T"], a["sk"], a["sv"], a["S"], a["gk"],
                                a["gv"], a["cap"], a["ss"], a["sl"], a["n"], a["hint"], a["Hq"], a["Hkv"], a["D"],
                                a["scale"], a["out"], a["odt"], a["lse"], a["splits"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(T=3), -1),                         # fewer tail tokens than query rows
    (dict(Lq=-1), -1),
    (dict(n=2049), -1),                      # segment table too long
    (dict(n=-1), -1),
    (dict(hint=-1), -1),
    (dict(Hq=3, Hkv=2), -1),
    (dict(D=80), -2),
    (dict(odt=5), -2),
    (dict(scale=float("inf")), -1),
    (dict(splits=-1), -1),
    (dict(q=None), -1),
    (dict(tk=None), -1),
    (dict(sk=None), -1),
    (dict(ss=None), -1),
    (dict(gk=None), -1),
    (dict(q=MIS), -4),
    (dict(ss=A + 0x700004), -4),
    (dict(sl=A + 0x701002), -4),
    (dict(out=A + 0x500000), -1),            # output inside the store
    (dict(lse=A + 0x700000), -1),            # lse over the segment table
    (dict(n=2048, cap=1 << 20), -1),         # possible gathered keys beyond 2^30
    (dict(splits=4, Lq=4), -5),              # split without a workspace
])
def test_gather_rejects_bad_arguments(kw, status):
    assert _gather(**kw) == status


def test_gather_zero_rows_is_a_no_op():
    assert _gather(Lq=0) == 0


def _gather_noalloc(**kw):
    a = dict(q=A, Lq=4, tk=A + 0x100000, tv=A + 0x200000, T=6, sk=A + 0x300000, sv=A + 0x400000, S=8,
             gk=A + 0x500000, gv=A + 0x600000, cap=500, ss=A + 0x700000, sl=A + 0x701000, n=3, hint=100,
             Hq=2, Hkv=1, D=64, scale=0.0, out=B, odt=1, lse=None, splits=0)
    a.update(kw)
    return lib.vico_gather_attn_noalloc(a["q"], a["Lq"], a["tk"], a["tv"], a["T"], a["sk"], a["sv"], a["S"],
                                        a["gk"], a["gv"], a["cap"], a["ss"], a["sl"], a["n"], a["hint"], a["Hq"],
                                        a["Hkv"], a["D"], a["scale"], a["out"], a["odt"], a["lse"], a["splits"],
                                        None)


@pytest.mark.parametrize("kw,status", [
    (dict(T=3), -1),
    (dict(D=80), -2),
    (dict(q=None), -1),
    (dict(q=MIS), -4),
    (dict(out=A + 0x500000), -1),
    (dict(n=2048, cap=1 << 20), -1),
])
def test_gather_noalloc_rejects_bad_arguments(kw, status):
    """Argument checks are those of vico_gather_attn, made before the library's
    array is looked up."""
    assert _gather_noalloc(**kw) == status


def test_gather_noalloc_rejects_work_beyond_its_array():
    """A plan needing more partials than the fixed array holds fails before any
    HIP call: 128 query rows at 28 heads, d 128, split 64 ways need 118 MB."""
    kw = dict(Lq=128, T=128, S=64, cap=200000, n=32, hint=20480, Hq=28, Hkv=4, D=128, splits=64,
              sk=A + (1 << 26), sv=A + (2 << 26), tk=A + (3 << 26), tv=A + (4 << 26), gk=A + (5 << 26),
              gv=A + (7 << 26), ss=A + (9 << 26), sl=A + (10 << 26), out=A + (11 << 26))
    wb = vico.vico_gather_plan(128, 128, 64, 200000, 32, 20480, 28, 4, 128, num_splits=64)[1]
    assert wb > vico.VICO_NOALLOC_SCRATCH_BYTES
    assert _gather_noalloc(**kw) == -7
    assert lib.vico_status_str(-7) != b"unknown status"


@pytest.mark.parametrize("Hq,Hkv,D", [(28, 4, 128), (16, 2, 128), (64, 8, 128), (7, 1, 64)])
def test_gather_noalloc_array_holds_every_default_plan(Hq, Hkv, D):
    """With the library's own split every query length fits the array."""
    for Lq in list(range(1, 300)) + list(range(300, 4097, 37)):
        wb = vico.vico_gather_plan(Lq, Lq, 64, 200000, 32, 20480, Hq, Hkv, D)[1]
        assert wb <= vico.VICO_NOALLOC_SCRATCH_BYTES, (Lq, wb)


def test_gather_noalloc_zero_rows_is_a_no_op():
    assert _gather_noalloc(Lq=0) == 0


def test_noalloc_scratch_size_matches_the_header():
    src = open(vico.load_library.__globals__["HEADER"]).read()
    assert "#define VICO_NOALLOC_SCRATCH_BYTES (64ll << 20)" in src
    assert vico.VICO_NOALLOC_SCRATCH_BYTES == 64 << 20


def test_gather_plan_parts():
    # 7B heads, 32-token query, ~20k gathered keys: 4 KV heads x 64 parts fill the CUs
    assert vico.vico_gather_plan(32, 32, 64, 200000, 32, 20480, 28, 4, 128)[0] == 64
    # decode step over a short window: few key tiles, few parts
    p, wb = vico.vico_gather_plan(1, 1, 0, 256, 2, 256, 2, 1, 64)
    assert p == 1 and wb == 0
    p, wb = vico.vico_gather_plan(1, 1, 0, 256, 2, 256, 2, 1, 64, num_splits=3)
    assert p == 3 and wb == 256 * ((3 * 2 * 1 * 64 * 4 + 255) // 256) + 3 * 2 * 4
    assert vico.vico_gather_plan(1, 1, 0, 256, 2, 256, 2, 1, 64, num_splits=500)[0] == 64


# ---------------------------------------------------------------- options and the chunk-granular window

def test_unknown_attention_flags_are_rejected():
    st = lib.vico_chunk_prefill_attn_ex(A, A + 0x100000, A + 0x200000, 64, A + 0x300000, A + 0x400000, 16,
                                        A + 0x500000, A + 0x600000, 256, 456, 256, 2, 1, 64, 0.0, B, 1, None, 0, 4,
                                        None, 0, None)
    assert st == -1
    assert vico.vico_attn_plan(64, 16, 256, 456, 256, 2, 1, 64, 0, 1) == vico.vico_attn_plan(64, 16, 256, 456,
                                                                                              256, 2, 1, 64, 0, 0)
    with pytest.raises(vico.VicoError):
        vico.vico_attn_plan(64, 16, 256, 456, 256, 2, 1, 64, 0, 4)


@pytest.mark.parametrize("seed", range(5))
def test_acn_window_matches_oracle(seed):
    import numpy as np
    import oracle
    rng = np.random.default_rng(seed)
    starts = np.concatenate([[0], np.cumsum(rng.integers(0, 900, 40))])
    for t in range(len(starts)):
        for acn in (-1, 0, 1, 2, 4, 8, 100):
            assert vico.vico_acn_window(list(starts), t, acn) == oracle.acn_window(starts, t, acn)


def test_acn_window_rejects_bad_tables():
    arr = (ctypes.c_int64 * 3)(0, 10, 5)
    assert lib.vico_acn_window(arr, 3, 3, 1) == -1          # t outside the table
    assert lib.vico_acn_window(arr, 3, -1, 1) == -1
    assert lib.vico_acn_window(None, 3, 1, 1) == -1
    assert lib.vico_acn_window(arr, 3, 2, 1) == -1          # decreasing starts


@pytest.mark.parametrize("kw,status", [
    (dict(C=300, R=256, W=200), -3),                 # the appended chunk is longer than the ring
    (dict(rk=None, rv=None, W=0, H=0), -1),          # nothing to append to
    (dict(kc=A + 0x500000), -1),                     # the chunk's K inside the ring the append writes
    (dict(ws=A + 0x600000, wsb=1 << 30, splits=2), -1),   # the merge's workspace inside the ring
])
def test_attention_append_rejects_bad_arguments(kw, status):
    a = dict(q=A, kc=A + 0x100000, vc=A + 0x200000, C=64, sk=A + 0x300000, sv=A + 0x400000, S=16,
             rk=A + 0x500000, rv=A + 0x600000, R=256, H=456, W=256, Hq=2, Hkv=1, D=64, scale=0.0,
             out=B, odt=1, lse=None, splits=0, ws=None, wsb=0)
    a.update(kw)
    st = lib.vico_chunk_prefill_attn_ex(a["q"], a["kc"], a["vc"], a["C"], a["sk"], a["sv"], a["S"], a["rk"], a["rv"],
                                        a["R"], a["H"], a["W"], a["Hq"], a["Hkv"], a["D"], a["scale"], a["out"],
                                        a["odt"], a["lse"], a["splits"], vico.VICO_ATTN_APPEND, a["ws"], a["wsb"],
                                        None)
    assert st == status


def test_append_flag_is_accepted_by_the_plan():
    assert vico.vico_attn_plan(64, 16, 256, 456, 256, 2, 1, 64, 0, vico.VICO_ATTN_APPEND) == \
        vico.vico_attn_plan(64, 16, 256, 456, 256, 2, 1, 64)


def test_balanced_plan_counts_whole_chunks_when_bidirectional():
    # bidirectional rows all see the whole chunk: more key tiles, possibly more parts
    c = dict(chunk_len=600, sink_len=64, ring_slots=4596, hist_len=4596, window=4000, num_q_heads=8,
             num_kv_heads=2, head_dim=128, num_splits=vico.VICO_SPLIT_BALANCED)
    causal = vico.vico_attn_plan(**c)
    bidir = vico.vico_attn_plan(**c, flags=vico.VICO_ATTN_BIDIRECTIONAL)
    assert bidir[0] >= causal[0] >= 1


def _drop(**kw):
    a = dict(fr=A, B=2, C=4, nf=24, dm=64, tau=0.9, prev=None, keep=B, sim=B + 0x1000, out=B + 0x10000,
             idx=B + 0x100000, cnt=B + 0x200000, ws=None, wsb=0)
    a.update(kw)
    return lib.vico_temporal_drop(a["fr"], a["B"], a["C"], a["nf"], a["dm"], a["tau"], a["prev"], a["keep"],
                                  a["sim"], a["out"], a["idx"], a["cnt"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(C=0), -1), (dict(C=9), -1), (dict(nf=0), -1), (dict(dm=60), -1), (dict(B=-1), -1),
    (dict(tau=float("nan")), -1), (dict(fr=None), -1), (dict(keep=None), -1), (dict(idx=None), -1),
    (dict(cnt=None), -1), (dict(fr=MIS), -4), (dict(out=B + 0x10008), -4), (dict(idx=B + 0x100002), -4),
    (dict(keep=A + 0x100), -1),              # keep inside the frames
    (dict(out=B + 0x800), -1),               # out_tokens over sim
    (dict(ws=B + 0x300000, wsb=-8), -1),
    (dict(ws=B + 0x300000, wsb=351), -5),    # one byte short of the 352 the shape needs
    (dict(ws=B + 0x300004, wsb=4096), -4),   # control words are 8-byte aligned
    (dict(ws=B + 0x10, wsb=4096), -1),       # workspace over keep (48 bytes)
    (dict(ws=A + 0x40, wsb=4096), -1),       # workspace inside the frames
])
def test_temporal_drop_rejects_bad_arguments(kw, status):
    assert _drop(**kw) == status


def test_temporal_drop_of_no_chunks_is_a_no_op():
    assert _drop(B=0) == 0
    assert _drop(B=0, ws=B + 0x300000, wsb=0) == 0


def _ws(B, n_f):
    """A 128-byte line per chunk and an 8-byte word per tile of 4 positions."""
    return 128 * B + 8 * B * -(-n_f // 4)


@pytest.mark.parametrize("shape,want", [
    ((2, 4, 24, 64), _ws(2, 24)),
    ((16, 4, 256, 3584), _ws(16, 256)),
    ((3, 1, 40, 4096), _ws(3, 40)),          # C = 1 compares 2 rows: 8 units of 512 features fit
    ((3, 1, 40, 4104), 0),                   # 9 units per lane: two passes
    ((3, 4, 41, 4096), _ws(3, 41)),
    ((3, 5, 40, 3072), _ws(3, 40)),
    ((3, 5, 40, 3080), 0),
    ((3, 8, 40, 2048), _ws(3, 40)),
    ((3, 8, 40, 2056), 0),
    ((3, 4, 1024, 64), _ws(3, 1024)),
    ((3, 4, 1025, 64), 0),                   # more than 256 tiles per chunk
    ((256, 4, 24, 64), _ws(256, 24)),        # the most chunks one call takes
    ((257, 4, 24, 64), 0),
    ((0, 4, 24, 64), 0),
    ((2, 9, 24, 64), -1), ((2, 4, 24, 60), -1), ((-1, 4, 24, 64), -1), ((1 << 20, 8, 1 << 10, 8), -1),
])
def test_temporal_drop_workspace_bytes(shape, want):
    assert lib.vico_temporal_drop_workspace_bytes(*shape) == want


# ---- measurement helper library (libvico_bench.so, include/vico_bench.h)

def _bench_header_functions():
    import re
    from paper_2606_19849_amd.build import INCLUDE
    src = open(f"{INCLUDE}/vico_bench.h").read()
    src = re.sub(r"//[^\n]*", "", src)
    return sorted(set(re.findall(r"\b(vico_\w+)\s*\(", src)))


def test_bench_library_exports_its_header():
    from paper_2606_19849_amd.build import BENCH_LIB
    blib = ctypes.CDLL(BENCH_LIB)
    names = _bench_header_functions()
    assert names == ["vico_bench_mfma_peak"]
    for n in names:
        assert hasattr(blib, n)


@pytest.mark.parametrize("groups,iters,sink", [(0, 10, A), (4, 0, A), (4, 10, None), (-1, 10, A)])
def test_bench_mfma_peak_rejects_bad_arguments(groups, iters, sink):
    from paper_2606_19849_amd.build import BENCH_LIB
    fn = ctypes.CDLL(BENCH_LIB).vico_bench_mfma_peak
    fn.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int32
    assert fn(groups, iters, sink, None) == -1      # VICO_ERR_INVALID_ARG, before any HIP call


def test_tensor_size_limit_is_2_to_the_31_bytes():
    """K/V tensors are addressed through 32-bit buffer offsets: one d128 head of
    2^23 - 1 ring or store slots is the largest accepted, 2^23 slots (exactly
    2^31 bytes) is rejected."""
    R = (1 << 23) - 1
    assert vico.vico_attn_plan(64, 16, R, R + 777, R - 100000, 2, 1, 128)[0] >= 1
    with pytest.raises(vico.VicoError):
        vico.vico_attn_plan(64, 16, R + 1, R + 777, R - 100000, 2, 1, 128)
    assert vico.vico_gather_plan(2, 64, 16, R, 3, 10000, 7, 1, 128)[0] >= 1
    with pytest.raises(vico.VicoError):
        vico.vico_gather_plan(2, 64, 16, R + 1, 3, 10000, 7, 1, 128)
