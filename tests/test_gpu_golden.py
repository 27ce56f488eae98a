"""The HIP path on the fixtures of tests/golden/ (closed-form cases written
from the oracle by tests/golden/make_golden.py).

Attention with Q = 0: every logit is 0 on the GPU too, so every probability
is exactly 1, the sums of the small-integer V rows are exact in fp32, and
each output is the mean of the visible V rows up to fp32 rounding of one
division.  Token dropping on exact-cosine vectors: the decisions, retained
rows and count are integers and must match exactly on both schedules."""
import json
import os

import numpy as np
import pytest
import torch

import paper_2606_19849_amd as vico
from tests._gpu import dev

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def bf16_rows(base, n, heads, d):
    """[n, heads, d] bf16 with row i, column c = base + i + c (exact integers)."""
    v = torch.arange(d, dtype=torch.float32).repeat(n, heads, 1) + base
    v += torch.arange(n, dtype=torch.float32)[:, None, None]
    return v.to(torch.bfloat16).cuda()


@pytest.mark.parametrize("case", load("attention_uniform.json")["cases"], ids=lambda c: c["name"])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_attention_uniform_golden(case, out_dtype):
    Hq, Hkv, d, S, R, H, W, C = (case[k] for k in ("num_q_heads", "num_kv_heads", "head_dim", "sink_len", "ring_slots",
                                                   "hist_len", "window", "chunk_len"))
    zeros = lambda n, h: torch.zeros((n, h, d), dtype=torch.bfloat16, device="cuda")
    q = zeros(C, Hq)
    kc, vc = zeros(C, Hkv), bf16_rows(60, C, Hkv, d)
    sk, sv = zeros(S, Hkv), bf16_rows(100, S, Hkv, d)
    rk, rv = zeros(R, Hkv), zeros(R, Hkv)
    hist_v = bf16_rows(10, H, Hkv, d)
    for p in range(max(0, H - R), H):                    # the resident history, slot p mod R
        rv[p % R] = hist_v[p]
    parts, wb = vico.vico_attn_plan(C, S, R, H, W, Hq, Hkv, d)
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
    out = torch.empty((C, Hq, d), dtype=out_dtype, device="cuda")
    lse = torch.empty((Hq, C), dtype=torch.float32, device="cuda")
    vico.vico_chunk_prefill_attn(q, kc, vc, sk, sv, rk, rv, H, W, out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    want = np.asarray(case["out_column0"])[:, :, None] + np.arange(d)[None, None, :]
    got = out.float().cpu().numpy().astype(np.float64)
    if out_dtype == torch.float32:
        assert np.max(np.abs(got - want) / want) <= 2.0 ** -23      # one fp32 division
    else:
        assert np.max(np.abs(got - want) / want) <= 2.0 ** -8       # then one bf16 rounding
    assert np.allclose(lse.cpu().numpy(), case["lse"], rtol=2.0 ** -20, atol=0)


@pytest.mark.parametrize("case", load("gather_uniform.json")["cases"], ids=lambda c: c["name"])
@pytest.mark.parametrize("parts", [0, 1, 3])
def test_gather_uniform_golden(case, parts):
    Hq, Hkv, d, S, cap, T, Lq = (case[k] for k in ("num_q_heads", "num_kv_heads", "head_dim", "sink_len",
                                                   "store_slots", "tail_len", "q_len"))
    b = case["bases"]
    zeros = lambda n, h: torch.zeros((n, h, d), dtype=torch.bfloat16, device="cuda")
    q = zeros(Lq, Hq)
    tk, tv = zeros(T, Hkv), bf16_rows(b["tail"], T, Hkv, d)
    sk, sv = zeros(S, Hkv), bf16_rows(b["sink"], S, Hkv, d)
    gk, gv = zeros(cap, Hkv), bf16_rows(b["store"], cap, Hkv, d)
    ss = torch.tensor(case["table_start"], dtype=torch.int64, device="cuda")    # clipped by the library
    sl = torch.tensor(case["table_len"], dtype=torch.int32, device="cuda")
    hint = int(sum(case["seg_len"]))
    np_, wb = vico.vico_gather_plan(Lq, T, S, cap, len(case["table_start"]), hint, Hq, Hkv, d, num_splits=parts)
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
    out = torch.empty((Lq, Hq, d), dtype=torch.float32, device="cuda")
    lse = torch.empty((Hq, Lq), dtype=torch.float32, device="cuda")
    vico.vico_gather_attn(q, tk, tv, sk, sv, gk, gv, ss, sl, out, lse=lse, workspace=ws, keys_hint=hint,
                          num_splits=parts)
    torch.cuda.synchronize()
    want = np.asarray(case["out_column0"])[:, :, None] + np.arange(d)[None, None, :]
    got = out.cpu().numpy().astype(np.float64)
    tol = 2.0 ** -23 if np_ == 1 else 2.0 ** -20      # the merge of parts adds a few fp32 roundings
    assert np.max(np.abs(got - want) / want) <= tol
    assert np.allclose(lse.cpu().numpy(), case["lse"], rtol=2.0 ** -20, atol=0)


@pytest.mark.parametrize("schedule", ["two_pass", "single_pass"])
def test_drop_exact_cosines_golden(schedule):
    g = load("drop_exact_cosines.json")
    vec, frames, dm = g["vectors"], g["frames"], g["dm"]
    c, n_f = 3, len(frames[0])
    B = len(frames) // c
    z = np.zeros((B, c, n_f, dm), dtype=np.float32)
    for fi, row in enumerate(frames):
        for p, key in enumerate(row):
            z[fi // c, fi % c, p, :2] = vec[key]
    bits = (z.view(np.uint32) >> 16).astype(np.uint16)           # small integers: exact in bf16
    fr = dev(bits)
    nb = vico.vico_temporal_drop_workspace_bytes(B, c, n_f, dm)
    ws = torch.full((nb,), 0xFF, dtype=torch.uint8, device="cuda") if schedule == "single_pass" else None
    for case in g["cases"]:
        keep = torch.full((B, n_f), 7, dtype=torch.uint8, device="cuda")
        sim = torch.full((B, n_f), float("nan"), dtype=torch.float32, device="cuda")
        idx = torch.full((B * c * n_f,), -5, dtype=torch.int32, device="cuda")
        cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        out = torch.zeros((B * c * n_f, dm), dtype=torch.bfloat16, device="cuda")
        vico.vico_temporal_drop(fr, float(np.float32(case["tau"])), keep, idx, cnt, sim=sim, out_tokens=out,
                                workspace=ws)
        torch.cuda.synchronize()
        n = int(cnt.item())
        assert np.array_equal(keep.cpu().numpy(), np.asarray(case["keep"], dtype=np.uint8)), case["tau"]
        assert n == len(case["index"]) and idx.cpu().numpy()[:n].tolist() == case["index"]
        assert np.array_equal(out[:n].cpu().view(torch.int16).numpy().view(np.uint16),
                              bits.reshape(B * c * n_f, dm)[case["index"]])
        assert np.max(np.abs(sim.cpu().numpy() - np.asarray(case["sim"]))) <= (3 * dm + 8) * 2.0 ** -24
