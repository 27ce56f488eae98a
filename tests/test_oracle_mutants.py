"""Planted mistakes in the oracle must fail its pins.

Each mutant is the oracle's own source with one plausible slip (an index off
by one, a dropped term, a wrong sign, a swapped operand, a wrong head map)
executed as a separate module on the CPU.  The pins used here are the same
independent references as in test_oracle_pins.py: torch SDPA in float64, the
zero-query closed form, brute-force ring bookkeeping and the LSE identity.
"""
import math
import os
import types

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from synth import ChunkShape, make_chunk_inputs
from tests._util import to_f64

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def _load(name, replace=None):
    src = open(os.path.join(ORACLE_DIR, name)).read()
    if replace is not None:
        old, new = replace
        assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType("oracle_mutant_" + name[:-3])
    exec(compile(src, name, "exec"), mod.__dict__)
    return mod


SHAPES = [ChunkShape(7, 1, 16, 3, 64, 150, 37, 9), ChunkShape(4, 2, 8, 2, 32, 70, 20, 6)]


def _attention_pins_hold(mod) -> bool:
    """True iff the (possibly mutated) attention module passes the SDPA pin and the
    zero-query closed form on SHAPES."""
    for sh in SHAPES:
        x = to_f64(make_chunk_inputs(sh, seed=21, family="F2"))
        try:
            o, lse = mod.chunk_prefill_attention(**x)
        except Exception:
            return False
        S, C, wv = sh.sink_len, sh.chunk_len, sh.visible_window
        n = x["hist_k"].shape[0]
        k = np.concatenate([x["sink_k"], x["hist_k"][n - wv:], x["k_chunk"]], 0)
        v = np.concatenate([x["sink_v"], x["hist_v"][n - wv:], x["v_chunk"]], 0)
        mask = torch.ones(C, S + wv + C, dtype=torch.bool)
        mask[:, S + wv:] = torch.tril(torch.ones(C, C, dtype=torch.bool))
        t = lambda a: torch.from_numpy(a).permute(1, 0, 2)[None]
        ref = F.scaled_dot_product_attention(t(x["q"]), t(k), t(v), attn_mask=mask, enable_gqa=True)
        if not np.max(np.abs(o - ref[0].permute(1, 0, 2).numpy())) <= 1e-12:
            return False
        g = sh.num_q_heads // sh.num_kv_heads
        kk = torch.from_numpy(k).repeat_interleave(g, dim=1)
        z = torch.einsum("chd,lhd->hcl", torch.from_numpy(x["q"]), kk) / math.sqrt(sh.head_dim)
        ref_lse = torch.logsumexp(z.masked_fill(~mask[None], -math.inf), dim=-1).numpy()
        if not np.max(np.abs(lse - ref_lse)) <= 1e-12:
            return False
        x0 = dict(x, q=np.zeros_like(x["q"]))
        _, lse0 = mod.chunk_prefill_attention(**x0)
        want = np.log(S + wv + np.arange(C) + 1.0)
        if not np.max(np.abs(lse0 - want[None, :])) <= 1e-13:
            return False
    return True


ATTN_MUTANTS = {
    "window_off_by_one": ("hist_k[n - wv:n, kv]", "hist_k[n - wv - 1:n - 1, kv]"),
    "strict_causal": ("j[None, :] <= np.asarray(rows)", "j[None, :] < np.asarray(rows)"),
    "gqa_modulo": ("return h // g", "return h % num_kv_heads"),
    "scale_1_over_d": ("return 1.0 / math.sqrt(head_dim)", "return 1.0 / head_dim"),
    "sink_dropped": ("[sink_k[:, kv], hist_k", "[sink_k[:0, kv], hist_k"),
    "values_from_keys": ("(p @ vals)", "(p @ keys)"),
    "lse_sign": ("m_safe[:, 0] + np.log", "m_safe[:, 0] - np.log"),
    "window_ignores_bound": ("return min(window, hist_len)", "return hist_len"),
    "max_not_subtracted_consistently": ("p = np.exp(z - m_safe)", "p = np.exp(z - 2 * m_safe)"),
}


def test_unmutated_oracle_passes_the_pins():
    assert _attention_pins_hold(_load("attention.py"))


@pytest.mark.parametrize("name", sorted(ATTN_MUTANTS))
def test_attention_mutant_is_caught(name):
    assert not _attention_pins_hold(_load("attention.py", ATTN_MUTANTS[name]))


def _ring_pins_hold(mod) -> bool:
    R = 64
    lin = np.arange(300 * 2, dtype=np.int64).reshape(300, 2)
    ring = mod.RingModel(R, (2,), np.int64)
    H = 0
    for c in (17, 64, 5, 40, 33, 64, 1, 76 - 0):
        c = min(c, 300 - H)
        H = ring.append(lin[H:H + c], H)
        lo = max(0, H - R)
        if not np.array_equal(ring.buf[np.arange(lo, H) % R], lin[lo:H]):
            return False
        for w in (0, 1, 13, min(R, H)):
            w = min(w, H)
            if not np.array_equal(ring.gather(H, w), lin[H - w:H]):
                return False
    return True


RING_MUTANTS = {
    "append_slot_shift": ("self.buf[(hist_len + j) % self.slots]", "self.buf[(hist_len + j + 1) % self.slots]"),
    "gather_off_by_one": ("(hist_len - count + k) % self.slots", "(hist_len - count + k - 1) % self.slots"),
}


def test_unmutated_ring_passes():
    assert _ring_pins_hold(_load("ring.py"))


@pytest.mark.parametrize("name", sorted(RING_MUTANTS))
def test_ring_mutant_is_caught(name):
    assert not _ring_pins_hold(_load("ring.py", RING_MUTANTS[name]))


def _merge_pin_holds(attn_mod, merge_mod) -> bool:
    rng = np.random.default_rng(3)
    q, k, v = rng.standard_normal((9, 8)) * 2, rng.standard_normal((50, 8)) * 2, rng.standard_normal((50, 8))
    vis = np.ones((9, 50), bool)
    whole, wl = attn_mod.softmax_attention(q, k, v, vis, 0.3)
    parts = [attn_mod.softmax_attention(q, k, v, np.pad(vis[:, a:b], ((0, 0), (a, 50 - b))), 0.3)
             for a, b in ((0, 20), (20, 50))]
    mo, ml = merge_mod.lse_merge([p[0] for p in parts], [p[1] for p in parts])
    return np.max(np.abs(mo - whole)) <= 1e-12 and np.max(np.abs(ml - wl)) <= 1e-12


@pytest.mark.parametrize("mut", [None, ("w = np.exp(L - m_safe)", "w = np.exp(m_safe - L)"),
                                 ("m_safe + np.log(", "m_safe * np.log(")])
def test_merge_mutants(mut):
    holds = _merge_pin_holds(_load("attention.py"), _load("merge.py", mut))
    assert holds == (mut is None)


# ---------------------------------------------------------------- chunk-granular window, bidirectional option

def _acn_pins_hold(mod) -> bool:
    from tests.test_oracle_acn_pins import _eq4_reference, _stream
    try:
        for acn, causal in ((2, False), (1, True), (3, False)):
            lens, chunks, sk, sv = _stream(7, 4, 2, 16, 3, seed=acn + 30)
            ref_o, _ = _eq4_reference(lens, chunks, sk, sv, acn, causal)
            starts = np.concatenate([[0], np.cumsum(lens)])
            hk = np.concatenate([c[1] for c in chunks])
            hv = np.concatenate([c[2] for c in chunks])
            for t, c in enumerate(lens):
                H = int(starts[t])
                q, kc, vc = chunks[t]
                o, _ = mod.chunk_prefill_attention(q, kc, vc, sk, sv, hk[:H], hv[:H], H,
                                                   mod.acn_window(starts, t, acn), bidirectional=not causal)
                if np.max(np.abs(o - ref_o[H:H + c])) > 1e-12:
                    return False
    except Exception:
        return False
    return True


ACN_MUTANTS = {
    "bidirectional_ignored": ("            if not bidirectional:\n", "            if True:\n"),
    "acn_one_chunk_too_many": ("starts[t] - starts[max(0, t - acn)]", "starts[t] - starts[max(0, t - acn - 1)]"),
    "acn_counts_current_chunk": ("starts[t] - starts[max(0, t - acn)]", "starts[t] - starts[max(0, t - acn + 1)]"),
}


def test_unmutated_acn_passes():
    assert _acn_pins_hold(_load("attention.py"))


@pytest.mark.parametrize("name", sorted(ACN_MUTANTS))
def test_acn_mutant_is_caught(name):
    assert not _acn_pins_hold(_load("attention.py", ACN_MUTANTS[name]))


# ---------------------------------------------------------------- temporal token dropping

def _drop_pins_hold(mod) -> bool:
    import itertools
    from scipy.spatial.distance import cdist
    import oracle
    from synth import make_drop_frames
    from tests.test_oracle_drop_pins import _brute
    f64 = oracle.bf16_bits_to_f64
    try:
        for shape, tau in (((3, 4, 24, 64), 0.9), ((2, 3, 30, 32), 0.0)):
            z = f64(make_drop_frames(*shape, seed=sum(shape)))
            keep, _, index = mod.temporal_drop(z, tau)
            bk, bi = _brute(z, tau)
            if not (np.array_equal(keep, bk) and np.array_equal(index, bi)):
                return False
        z = f64(make_drop_frames(6, 1, 32, 96, seed=3))
        keep, _, index = mod.temporal_drop(z, 0.7)
        bk, bi = _brute(z, 0.7)
        if not (np.array_equal(keep, bk) and np.array_equal(index, bi)):
            return False
        z = np.zeros((1, 2, 1, 4))
        z[0, 0, 0, :2] = (3, 4)
        z[0, 1, 0, :2] = (4, 3)
        if not mod.temporal_drop(z, 0.96)[0][0, 0]:
            return False
        a, b = np.eye(3)[0], np.eye(3)[1]
        z = np.stack([a, (a + b) / np.sqrt(2), b])[None, :, None, :]
        if not mod.temporal_drop(z, 0.5)[0][0, 0]:
            return False
    except Exception:
        return False
    return True


DROP_MUTANTS = {
    "threshold_not_strict": ("drop &= s_ij > tau", "drop &= s_ij >= tau"),
    # "any pair exceeds" instead of "all pairs exceed"
    "any_pair_drops": ("drop &= s_ij > tau", "drop = (drop & (i > 0)) | (s_ij > tau)"),
    "neighbours_only": ("for j in range(i + 1, c):", "for j in range(i + 1, min(i + 2, c)):"),
    "anchor_dropped": ("if (c > 1 and f == 0) or keep[b, p]:", "if keep[b, p]:"),
    "compare_with_next_frame": ("before = z[b - 1, 0] if b > 0 else prev", "before = z[b + 1, 0] if b + 1 < B else prev"),
    "position_major_order": ("for f in range(c):\n            for p in range(n_f):", "for p in range(n_f):\n            for f in range(c):"),
}


def test_unmutated_drop_passes():
    assert _drop_pins_hold(_load("token_drop.py"))


@pytest.mark.parametrize("name", sorted(DROP_MUTANTS))
def test_drop_mutant_is_caught(name):
    assert not _drop_pins_hold(_load("token_drop.py", DROP_MUTANTS[name]))
