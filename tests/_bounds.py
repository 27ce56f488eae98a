"""Per-element error bounds of the GPU attention against the fp64 oracle.

Test infrastructure.  The bounds follow the arithmetic of the kernels, which
compute, for a query row,

    O = sum_j bf16(p_j) v_j / sum_j p_j,   p_j = exp2(fl(s_j * c) - m),

with fp32 logits s_j (bf16 products, fp32 sums over head_dim), fp32 row sums
of the unrounded p_j, bf16 round-to-nearest-even of p_j for the P.V product
and fp32 accumulation (the attention definition of Sec. 3, "LLM Prefilling
and Decoding").  Against the exact O = sum_j p_j v_j / l, l = sum_j p_j:

  * bf16 rounding of p_j (relative error |e_j| <= u8 = 2^-8, 8 significant
    bits) moves O by sum_j p_j e_j v_j / l, at most u8 * A with
    A = sum_j p_j |v_j| / l -- the oracle's attention over |V|;
  * fp32 logits: a relative error eta_j of p_j moves O by at most
    max|eta| * sum_j p_j |v_j - O| / l <= 2 * eta * A.  The dot product of
    d bf16 products errs by at most (d+1) * 2^-24 * |q| |k| (Cauchy-Schwarz
    bounds sum |q_i k_i| by |q| |k|), the scale constant and the FMA add
    2^-24 of the logit, the hardware exp2 one ulp;
  * fp32 accumulation of O and l over the keys, whatever the order of the
    additions inside the matrix cores: at most (n - 1) * 2^-24 relative for a
    sum of n terms, n = visible keys for O and half of them per lane for l
    (kappa * A), the division by l and the output rounding (bf16 output: half
    an ulp, u8 * |O|);
  * with the key range split into parts, the log-sum-exp merge weights carry
    the parts' LSE errors: another 2 * eta * A plus fp32 rounding per part.

The LSE (natural log) errs by at most the largest logit error plus the fp32
rounding of the row sum, of log2 and of the final scaling.

A second, statistical gate (`hoeffding`) treats the bf16 rounding errors as
independent, zero-mean and bounded: with w_j = p_j |v_j| / l and
sigma^2 = (u8^2 / 3) sum_j w_j^2 (computed from the oracle: attention with
the scale doubled over V^2 gives sum_j p_j^2 v_j^2 / sum_j p_j^2, and
exp(LSE_2s - 2 LSE) = sum p^2 / l^2), Hoeffding's inequality gives
P(|err| > k sigma) <= 2 exp(-k^2 / 6); k = 13.5 keeps the chance that any
of 10^7 elements exceeds it below 2e-6.  This is the gate that is tight for
the near-uniform rows of the literal N(0,1)/sqrt(d) inputs, where the
worst case (all roundings aligned) is far from what happens.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

import oracle
from oracle.attention import default_scale

U8 = 2.0 ** -8      # bf16 unit roundoff
U24 = 2.0 ** -24    # fp32 unit roundoff
HOEFFDING_K = 13.5


@dataclass
class Bound:
    A: np.ndarray               # [rows, heads, d]: sum_j p_j |v_j| / l
    eta: np.ndarray             # [rows, heads]: relative error of a probability from fp32 logits and exp2
    dz: np.ndarray              # [heads, rows]: logit error bound in nats
    nkeys: int                  # largest visible key count of a row
    parts: int = 1              # key-range parts merged by log-sum-exp
    sigma: np.ndarray | None = None   # [rows, heads, d]: Hoeffding scale of the bf16 rounding error

    def _coef(self):
        kappa = (1.5 * self.nkeys + 64.0) * U24
        merge = (2.0 * self.eta[..., None] + self.parts * 2.0 ** -21) if self.parts > 1 else 0.0
        return U8 + 2.0 * self.eta[..., None] + kappa + merge

    def f32(self, ref):
        """Worst-case bound of |O_gpu - O| per element, fp32 output."""
        return self._coef() * self.A + 4.0 * U24 * np.abs(ref) + 1e-30

    def bf16(self, ref):
        """bf16 output: the fp32 bound plus the output rounding (half an ulp)."""
        b = self.f32(ref)
        return b + U8 * (np.abs(ref) + b)

    def lse(self, ref_lse):
        return (self.dz + (0.5 * self.nkeys + 64.0) * U24 + (40.0 + 2.0 * np.abs(ref_lse)) * 2.0 ** -22
                + self.parts * 2.0 ** -20)

    def hoeffding(self, ref):
        """Statistical bound: HOEFFDING_K * sigma plus the fp32 worst-case terms."""
        assert self.sigma is not None
        fp32 = (self._coef() - U8) * self.A + 4.0 * U24 * np.abs(ref)
        return HOEFFDING_K * self.sigma + fp32 + 1e-30


def _eta_dz(qn, kmax, scale, d, exact_dot=False):
    """qn [rows, heads] row norms of Q; kmax [heads] largest key norm seen by the head.
    exact_dot: Q and K are small integers, so every partial sum of a dot product
    is an integer below 2^24 and exact in fp32; only the scaling rounds."""
    dot = 0.0 if exact_dot else (d + 1) * U24
    dz = scale * qn * kmax[None, :] * (dot + 3 * U24) + 128.0 * U24
    return dz + 2.0 ** -22, dz.T


def _sigma(o2, lse2, lse):
    # sum_j p_j^2 v_j^2 / l^2 = O_2 * exp(LSE_2 - 2 LSE)
    r = np.exp(lse2 - 2.0 * lse).T[..., None]
    return (U8 / math.sqrt(3.0)) * np.sqrt(np.maximum(o2, 0.0) * r)


def chunk_bound(x, rows=None, heads=None, bidirectional=False, scale=None, parts=1, sigma=False, exact_dot=False):
    """Bound for the chunk-prefill attention; x = oracle inputs (tests._util.to_f64)."""
    q = x["q"]
    C, Hq, d = q.shape
    Hkv = x["k_chunk"].shape[1]
    g = Hq // Hkv
    rows = np.arange(C) if rows is None else np.asarray(rows)
    heads = np.arange(Hq) if heads is None else np.asarray(heads)
    s = default_scale(d) if scale is None else scale
    kw = dict(rows=rows, heads=heads, bidirectional=bidirectional, scale=s)
    xa = dict(x, v_chunk=np.abs(x["v_chunk"]), sink_v=np.abs(x["sink_v"]), hist_v=np.abs(x["hist_v"]))
    A, _ = oracle.chunk_prefill_attention(**xa, **kw)
    wv = oracle.visible_window(x["hist_len"], x["window"])
    n = x["hist_k"].shape[0]
    keys = np.concatenate([x["sink_k"], x["hist_k"][n - wv:n], x["k_chunk"]], axis=0)      # [L, Hkv, d]
    kmax = np.sqrt((keys ** 2).sum(-1)).max(axis=0)                                         # [Hkv]
    qn = np.sqrt((q[rows][:, heads] ** 2).sum(-1))                                           # [rows, heads]
    eta, dz = _eta_dz(qn, kmax[heads // g], s, d, exact_dot)
    nkeys = x["sink_k"].shape[0] + wv + C
    b = Bound(A, eta, dz, nkeys, parts)
    if sigma:
        _, lse = oracle.chunk_prefill_attention(**x, **kw)
        x2 = dict(x, v_chunk=x["v_chunk"] ** 2, sink_v=x["sink_v"] ** 2, hist_v=x["hist_v"] ** 2)
        o2, lse2 = oracle.chunk_prefill_attention(**x2, **dict(kw, scale=2.0 * s))
        b.sigma = _sigma(o2, lse2, lse)
    return b


def gather_bound(q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len, heads=None,
                 scale=None, parts=1, sigma=False):
    """Bound for the gathered-query attention (all float64 oracle inputs)."""
    Lq, Hq, d = q.shape
    Hkv = tail_k.shape[1]
    g = Hq // Hkv
    heads = np.arange(Hq) if heads is None else np.asarray(heads)
    s = default_scale(d) if scale is None else scale
    A, _ = oracle.gather_attention(q, tail_k, np.abs(tail_v), sink_k, np.abs(sink_v), store_k, np.abs(store_v),
                                   seg_start, seg_len, scale=s, heads=heads)
    segs = [store_k[a:a + m] for a, m in zip(seg_start, seg_len)]
    keys = np.concatenate([sink_k] + segs + [tail_k], axis=0)
    kmax = np.sqrt((keys ** 2).sum(-1)).max(axis=0)
    qn = np.sqrt((q[:, heads] ** 2).sum(-1))
    eta, dz = _eta_dz(qn, kmax[heads // g], s, d)
    nkeys = keys.shape[0]
    b = Bound(A, eta, dz, nkeys, parts)
    if sigma:
        _, lse = oracle.gather_attention(q, tail_k, tail_v, sink_k, sink_v, store_k, store_v, seg_start, seg_len,
                                         scale=s, heads=heads)
        o2, lse2 = oracle.gather_attention(q, tail_k, tail_v ** 2, sink_k, sink_v ** 2, store_k, store_v ** 2,
                                           seg_start, seg_len, scale=2.0 * s, heads=heads)
        b.sigma = _sigma(o2, lse2, lse)
    return b
