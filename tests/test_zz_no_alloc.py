"""vico_gather_attn_noalloc (the allocation-free variant of vico_gather_attn,
for callers that cannot allocate) against vico_gather_attn with a caller
workspace: the same kernels and the same plan, so outputs and LSE must agree
bit for bit.  Two calls in a row on the library's shared array, the second
smaller than the first, so the second runs over what the first left there."""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2606_19849_amd as vico
from synth import QUERY_CONFIGS, QueryShape, make_query_inputs
from tests._bounds import gather_bound
from tests._gpu import check_f32, dev

pytestmark = pytest.mark.gpu

f64 = oracle.bf16_bits_to_f64


class Case:
    def __init__(self, shape: QueryShape, seed: int, chunks, q_rows: int):
        qi = make_query_inputs(shape, seed=seed, family="F2")
        self.qi, self.sh, self.Lq = qi, shape, q_rows
        k, v = qi.store_kv()
        self.k_np, self.v_np = k, v
        self.q = dev(qi.q)[-q_rows:].contiguous()
        self.tk, self.tv = dev(qi.tail_k), dev(qi.tail_v)
        self.sk, self.sv = dev(qi.sink_k), dev(qi.sink_v)
        self.gk, self.gv = dev(k), dev(v)
        self.st, self.ln = oracle.chunk_segments(np.asarray(chunks), qi.chunk_start, qi.chunk_len)
        self.ss = torch.from_numpy(self.st.astype(np.int64)).cuda()
        self.sl = torch.from_numpy(self.ln.astype(np.int32)).cuda()
        self.hint = int(self.ln.sum())

    def buffers(self, dtype):
        sh = self.sh
        return (torch.full((self.Lq, sh.num_q_heads, sh.head_dim), 7.0, dtype=dtype, device="cuda"),
                torch.full((sh.num_q_heads, self.Lq), 7.0, dtype=torch.float32, device="cuda"))

    def plan(self, splits=0):
        sh = self.sh
        return vico.vico_gather_plan(self.Lq, sh.tail_len, sh.sink_len, self.gk.shape[0], len(self.st), self.hint,
                                     sh.num_q_heads, sh.num_kv_heads, sh.head_dim, splits)

    def with_workspace(self, dtype, splits=0):
        out, lse = self.buffers(dtype)
        wb = self.plan(splits)[1]
        ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
        vico.vico_gather_attn(self.q, self.tk, self.tv, self.sk, self.sv, self.gk, self.gv, self.ss, self.sl, out,
                              lse=lse, workspace=ws, keys_hint=self.hint, num_splits=splits)
        return out, lse

    def noalloc(self, out, lse, splits=0):
        vico.vico_gather_attn_noalloc(self.q, self.tk, self.tv, self.sk, self.sv, self.gk, self.gv, self.ss,
                                      self.sl, out, lse=lse, keys_hint=self.hint, num_splits=splits)

    def oracle_check(self, out, lse, parts):
        qi = self.qi
        args = (f64(qi.q)[-self.Lq:], f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k), f64(qi.sink_v),
                f64(self.k_np), f64(self.v_np), self.st, self.ln)
        ro, rl = oracle.gather_attention(*args)
        check_f32(out.cpu().numpy().astype(np.float64), ro, gather_bound(*args, parts=parts),
                  lse.cpu().numpy().astype(np.float64), rl)


# 7B heads: a 32-row query over 32 chunks (the plan splits the keys 64 ways:
# 29.6 MB of partials), then a decode step over 3 chunks (8 parts, 0.1 MB).
BIG = dataclasses.replace(QUERY_CONFIGS["q_7b"], num_chunks=40)
SMALL = dataclasses.replace(QUERY_CONFIGS["q_7b"], num_chunks=8, tail_len=64)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_noalloc_matches_the_workspace_entry_point_twice(dtype):
    first = Case(BIG, seed=41, chunks=range(4, 36), q_rows=32)
    second = Case(SMALL, seed=42, chunks=[1, 4, 6], q_rows=1)
    assert first.plan()[1] > second.plan()[1] > 0
    ref1 = first.with_workspace(dtype)
    ref2 = second.with_workspace(dtype)
    o1, l1 = first.buffers(dtype)
    o2, l2 = second.buffers(dtype)
    first.noalloc(o1, l1)
    second.noalloc(o2, l2)
    torch.cuda.synchronize()
    assert torch.equal(o1, ref1[0]) and torch.equal(l1, ref1[1])
    assert torch.equal(o2, ref2[0]) and torch.equal(l2, ref2[1])
    if dtype == torch.float32:
        first.oracle_check(o1, l1, first.plan()[0])
        second.oracle_check(o2, l2, second.plan()[0])


def test_noalloc_explicit_splits_and_unsplit():
    """An explicit split count (partials in the array) and one part (no
    partials: the array is not touched) agree with the workspace path."""
    c = Case(dataclasses.replace(QUERY_CONFIGS["q_gqa7"]), seed=43, chunks=[0, 3, 5, 8], q_rows=4)
    for splits in (7, 1, 3):
        ref = c.with_workspace(torch.float32, splits)
        o, l = c.buffers(torch.float32)
        c.noalloc(o, l, splits)
        torch.cuda.synchronize()
        assert torch.equal(o, ref[0]) and torch.equal(l, ref[1]), splits


def test_noalloc_rejects_a_plan_beyond_its_array():
    c = Case(dataclasses.replace(QUERY_CONFIGS["q_7b"], num_chunks=4, q_len=128, tail_len=128), seed=44,
             chunks=[0, 1, 2, 3], q_rows=128)
    assert c.plan(64)[1] > vico.VICO_NOALLOC_SCRATCH_BYTES
    o, l = c.buffers(torch.float32)
    with pytest.raises(vico.VicoError) as e:
        c.noalloc(o, l, splits=64)
    assert e.value.status == -7
    torch.cuda.synchronize()
    assert bool(torch.all(o == 7.0)) and bool(torch.all(l == 7.0))     # nothing was written
