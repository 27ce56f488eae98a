"""Planted mistakes in the retrieval oracle must fail its pins.

Each mutant is oracle/retrieval.py with one plausible slip, executed as a
separate module.  The pins are independent references: statistics.fmean,
scipy's cosine distance, brute-force subset selection and torch SDPA in
float64 over keys listed slot by slot.
"""
import math
import os
import statistics
import types

import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle
from synth import QUERY_CONFIGS, make_query_inputs, make_tokens
from tests.test_oracle_retrieval_pins import _brute_force_select, _sdpa_reference

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def _load(replace=None):
    src = open(os.path.join(ORACLE_DIR, "retrieval.py")).read()
    src = src.replace("from .attention import", "from oracle.attention import")
    if replace is not None:
        old, new = replace
        assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType("oracle_mutant_retrieval")
    exec(compile(src, "retrieval.py", "exec"), mod.__dict__)
    return mod


def _pins_hold(R) -> bool:
    f64 = oracle.bf16_bits_to_f64
    try:
        x = f64(make_tokens(37, 64, seed=3))
        if np.max(np.abs(R.token_mean(x) - [statistics.fmean(x[:, j]) for j in range(64)])) > 1e-14:
            return False
        rng = np.random.default_rng(0)
        q, c = rng.standard_normal(48), rng.standard_normal((30, 48)) * np.arange(1, 31)[:, None]
        if np.max(np.abs(R.cosine_scores(q, c) - (1.0 - cdist(q[None], c, metric="cosine")[0]))) > 1e-13:
            return False
        for seed in range(6):
            s = np.round(np.random.default_rng(seed).uniform(-1, 1, 9), 1)
            for k in (1, 3, 5):
                if list(R.select_chunks(s, k)) != _brute_force_select(s, k):
                    return False
        s = np.array([0.3, 0.5, 0.3, -0.2, 0.1])
        if list(R.select_chunks(s, 4, 0.3)) != _brute_force_select(s, 4, 0.3):
            return False
        for name in ("q_tiny", "q_gqa7"):
            qi = make_query_inputs(QUERY_CONFIGS[name], seed=1, family="F2")
            sel = R.select_chunks(np.arange(qi.shape.num_chunks)[::-1] % 5, qi.shape.top_k)
            st, ln = R.chunk_segments(sel, qi.chunk_start, qi.chunk_len)
            stk, stv = (f64(a) for a in qi.store_kv())
            out, lse = R.gather_attention(f64(qi.q), f64(qi.tail_k), f64(qi.tail_v), f64(qi.sink_k),
                                          f64(qi.sink_v), stk, stv, st, ln)
            ro, rl = _sdpa_reference(qi, st, ln)
            if np.max(np.abs(out - ro)) > 1e-12 or np.max(np.abs(lse - rl)) > 1e-12:
                return False
    except Exception:
        return False
    return True


MUTANTS = {
    "mean_over_L_minus_1": ("/ x.shape[0]", "/ (x.shape[0] - 1)"),
    "cosine_no_chunk_norm": ("np.sqrt(np.sum(c * c, axis=1)) * math.sqrt", "math.sqrt"),
    "cosine_query_norm_squared": ("math.sqrt(float(q @ q))", "float(q @ q)"),
    "ties_prefer_later_chunk": ("key=lambda i: (-s[i], i)", "key=lambda i: (-s[i], -i)"),
    "threshold_strict": ("s[i] >= min_score", "s[i] > min_score"),
    "top_k_of_ascending_scores": ("key=lambda i: (-s[i], i)", "key=lambda i: (s[i], i)"),
    "segment_shifted_by_one": ("store[int(a):int(a) + int(n), kv]", "store[int(a) + 1:int(a) + int(n) + 1, kv]"),
    "tail_strictly_causal": ("tail_pos[None, :] <= row_pos[:, None]", "tail_pos[None, :] < row_pos[:, None]"),
    "rows_at_tail_start": ("row_pos = T - Lq + np.arange(Lq)", "row_pos = np.arange(Lq)"),
    "gqa_modulo": ("kv = kv_head_of(int(h), Hq, Hkv)", "kv = int(h) % Hkv"),
    "sink_dropped": ("keys = np.concatenate([sink_k[:, kv], gk", "keys = np.concatenate([sink_k[:0, kv], gk"),
}


def test_unmutated_retrieval_oracle_passes():
    assert _pins_hold(_load())


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_retrieval_mutant_is_caught(name):
    assert not _pins_hold(_load(MUTANTS[name]))
