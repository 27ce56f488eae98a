"""GPU-test helpers: move synthetic bf16 bits to the device, call the library
through the binding, and compare with the oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2606_19849_amd as vico
from synth import ChunkInputs
from tests._util import ring_from_inputs, to_f64


def dev(bits: np.ndarray) -> torch.Tensor:
    """bf16 bit patterns (uint16) -> contiguous bfloat16 CUDA tensor."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def bits_of(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


class DeviceChunk:
    def __init__(self, inp: ChunkInputs):
        sh = inp.shape
        self.inp = inp
        self.q, self.kc, self.vc = dev(inp.q), dev(inp.k_chunk), dev(inp.v_chunk)
        self.sk = dev(inp.sink_k) if sh.sink_len else None
        self.sv = dev(inp.sink_v) if sh.sink_len else None
        rk, rv = ring_from_inputs(inp)
        self.rk = dev(rk) if sh.ring_slots else None
        self.rv = dev(rv) if sh.ring_slots else None

    def attention(self, out_dtype=torch.float32, num_splits=0, with_lse=True, flags=0, scale=0.0):
        sh = self.inp.shape
        out = torch.empty((sh.chunk_len, sh.num_q_heads, sh.head_dim), dtype=out_dtype, device="cuda")
        lse = torch.empty((sh.num_q_heads, sh.chunk_len), dtype=torch.float32, device="cuda") if with_lse else None
        _, wb = vico.vico_attn_plan(sh.chunk_len, sh.sink_len, sh.ring_slots, sh.hist_len, sh.window,
                                    sh.num_q_heads, sh.num_kv_heads, sh.head_dim, num_splits, flags)
        ws = torch.empty(wb, dtype=torch.uint8, device="cuda") if wb else None
        vico.vico_chunk_prefill_attn(self.q, self.kc, self.vc, self.sk, self.sv, self.rk, self.rv,
                                     sh.hist_len, sh.window, out, lse=lse, workspace=ws, num_splits=num_splits,
                                     softmax_scale=scale, flags=flags)
        torch.cuda.synchronize()
        o = out.float().cpu().numpy().astype(np.float64)
        l = lse.cpu().numpy().astype(np.float64) if with_lse else None
        return o, l


def oracle_result(inp: ChunkInputs, rows=None, heads=None, bidirectional=False, scale=None):
    return oracle.chunk_prefill_attention(**to_f64(inp), rows=rows, heads=heads, bidirectional=bidirectional,
                                          scale=scale)


def check_f32(o, ref, lse=None, ref_lse=None, max_abs=1e-2, mean_abs=1e-3, lse_abs=1e-3):
    """Binding tolerance on O(1)-scaled outputs (fp32 output path).

    The probabilities are rounded to bf16 (relative error up to 2^-9 per
    weight), so an output's error carries the size of the values it averages;
    the max-abs bound applies per unit of output magnitude: |err| <= max_abs *
    max(1, |ref|).  Mean-abs is bounded absolutely."""
    assert np.all(np.isfinite(o))
    err = np.abs(o - ref)
    excess = err - max_abs * np.maximum(1.0, np.abs(ref))
    assert excess.max() <= 0, f"max-abs {err.max():.3e} (largest excess {excess.max():.3e})"
    assert err.mean() <= mean_abs, f"mean-abs {err.mean():.3e}"
    if lse is not None:
        le = np.abs(lse - ref_lse)
        assert le.max() <= lse_abs, f"lse max-abs {le.max():.3e}"
    return err.max(), err.mean()


def check_bf16(o, ref, max_abs=1e-2, mean_abs=1e-3):
    """bf16 output: the fp32 tolerance plus half a bf16 ulp of rounding (2^-8 relative)."""
    assert np.all(np.isfinite(o))
    err = np.abs(o - ref)
    bound = max_abs * np.maximum(1.0, np.abs(ref)) + np.abs(ref) * 2.0 ** -8
    assert np.all(err <= bound), f"max excess {np.max(err - bound):.3e}"
    assert err.mean() <= mean_abs + np.mean(np.abs(ref)) * 2.0 ** -9, f"mean-abs {err.mean():.3e}"


def check_relative(o, ref, rel_fro=5e-3):
    """Scale-free check for the N(0,1)/sqrt(d) inputs, whose outputs are ~1e-3 in size."""
    assert np.all(np.isfinite(o))
    r = np.linalg.norm(o - ref) / np.linalg.norm(ref)
    assert r <= rel_fro, f"relative Frobenius error {r:.3e}"
    return r
