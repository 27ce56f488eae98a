"""Writes the small fixtures of tests/golden/ from the oracle alone.

    python tests/golden/make_golden.py

Each fixture is a case whose result also has a closed form (tests/test_golden.py
checks both against the stored values).  The paper prints no worked numeric
example, so these are the stored values.

  attention_uniform.json
      Chunk prefill with Q = 0, so every visible logit is 0 and each output
      row is the plain mean of the visible V rows; V rows encode their key's
      position.  The mean names exactly which sink, window and chunk keys a
      row sees: the bounded visible set of Sec. 3 ("LLM Prefilling and
      Decoding"), token-granular with the causal chunk, read through a ring
      that has wrapped.  LSE = ln(number of visible keys).
  gather_uniform.json
      Short-query attention over sink ++ store segments ++ causal tail with
      Q = 0 (the query-time attention of Sec. 3 over the retrieved chunks):
      each output row is the mean of the V rows of the sink, of the store
      slots the segments list (in table order, an empty segment included)
      and of tail tokens 0 .. T-Lq+i.  A 3-row query and a decode step.
      The table handed to the library ("table_start"/"table_len") also has
      segments reaching outside the store, which the library clips to it;
      the oracle gets the clipped table ("seg_start"/"seg_len").
  acn_windows.json
      The chunk-granular window of Eq. (4): the history tokens of chunks
      t-acn .. t-1 for a ragged table of chunk starts.
  drop_exact_cosines.json
      Temporal token dropping (Sec. 3, "Token Dropping") on vectors whose
      pairwise cosines are exact rationals (3-4-5 and 5-12-13 triangles),
      against thresholds on both sides of them: keep flags, smallest
      cosines and the retained rows in stream order.
"""
from __future__ import annotations

import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402


def attention_uniform_cases():
    cases = []
    for name, (Hq, Hkv, d, S, R, H, W, C) in {
        "bounded_wrapped": (2, 1, 64, 2, 4, 6, 3, 3),     # window positions 3..5 in slots 3, 0, 1
        "full_history": (4, 2, 64, 3, 8, 5, -1, 4),       # every history token visible
        "no_history": (2, 2, 128, 1, 4, 0, 4, 5),         # sink and chunk only
    }.items():
        # V rows: column c of the key at linear key position k holds base(k) + c,
        # base = 100 + s for sink s, 10 + p for history position p, 60 + j for
        # chunk token j (small integers: exact in bf16)
        def rows(base, n, heads):
            v = np.zeros((n, heads, d))
            for i in range(n):
                v[i] = base + i + np.arange(d)[None, :]
            return v

        sink_v = rows(100, S, Hkv)
        hist_v = rows(10, H, Hkv)
        chunk_v = rows(60, C, Hkv)
        zeros = lambda n: np.zeros((n, Hkv, d))
        q = np.zeros((C, Hq, d))
        out, lse = oracle.chunk_prefill_attention(q, zeros(C), chunk_v, zeros(S), sink_v, zeros(H), hist_v, H, W)
        cases.append({
            "name": name,
            "num_q_heads": Hq, "num_kv_heads": Hkv, "head_dim": d, "sink_len": S, "ring_slots": R,
            "hist_len": H, "window": W, "chunk_len": C,
            "value_rule": "v[key][kv][c] = base + index + c; base 100 (sink s), 10 (history position p), 60 (chunk j)",
            "out_column0": out[:, :, 0].tolist(),          # column c is column 0 + c
            "lse": lse.tolist(),
        })
    return {"citation": "Sec. 3, LLM Prefilling and Decoding (bounded visible set); Eq. (4) vision rows",
            "cases": cases}


def gather_uniform_cases():
    cases = []
    for name, (Hq, Hkv, d, S, cap, segs, T, Lq, bases) in {
        "query": (4, 2, 64, 2, 48, [(30, 5), (2, 7), (15, 0), (40, 12), (-3, 5), (50, 4), (10, -2)], 6, 3,
                  (100, 120, 30)),
        "decode": (2, 1, 128, 1, 20, [(0, 20)], 4, 1, (10, 20, 60)),
    }.items():
        b_sink, b_store, b_tail = bases

        def rows(base, n):
            v = np.zeros((n, Hkv, d))
            for i in range(n):
                v[i] = base + i + np.arange(d)[None, :]
            return v

        z = lambda n: np.zeros((n, Hkv, d))
        # the library's contract for a table entry: slots [max(0, a), min(a + n, cap)), empty if none
        clipped = [(max(0, a), min(a + n, cap) - max(0, a)) if min(a + n, cap) > max(0, a) else (0, 0)
                   for a, n in segs]
        starts = [a for a, _ in clipped]
        lens = [n for _, n in clipped]
        out, lse = oracle.gather_attention(np.zeros((Lq, Hq, d)), z(T), rows(b_tail, T), z(S), rows(b_sink, S),
                                           z(cap), rows(b_store, cap), starts, lens)
        cases.append({
            "name": name, "num_q_heads": Hq, "num_kv_heads": Hkv, "head_dim": d, "sink_len": S,
            "store_slots": cap, "table_start": [a for a, _ in segs], "table_len": [n for _, n in segs],
            "seg_start": starts, "seg_len": lens, "tail_len": T, "q_len": Lq,
            "bases": {"sink": b_sink, "store": b_store, "tail": b_tail},
            "value_rule": "v[key][kv][c] = base + index + c (index: sink s, store slot, tail token t)",
            "out_column0": out[:, :, 0].tolist(),
            "lse": lse.tolist(),
        })
    return {"citation": "Sec. 3, query-time decoding (attention over the retrieved chunks)", "cases": cases}


def acn_cases():
    starts = [0, 300, 300, 1324, 1580, 2604, 2860, 3116]     # ragged chunk lengths, one empty chunk
    table = []
    for acn in (-1, 0, 1, 2, 5):
        table.append({"acn": acn, "windows": [oracle.acn_window(starts, t, acn) for t in range(len(starts))]})
    return {"citation": "Eq. (4) (vision rows: chunks t-acn .. t)", "chunk_starts": starts, "table": table}


def drop_cases():
    # 2 chunks of 3 frames of 4 positions, dm 8; the first two features carry
    # the vectors, the rest are zero
    vec = {
        "a": (3, 4), "b": (4, 3), "c": (5, 0), "d": (5, 12), "e": (12, 5), "z": (0, 0),
    }
    frames = [
        ["a", "a", "c", "z"],      # frame 0 (anchor) of chunk 0
        ["a", "b", "c", "z"],
        ["a", "a", "d", "z"],
        ["d", "b", "a", "c"],      # chunk 1
        ["d", "a", "a", "c"],
        ["e", "a", "b", "c"],
    ]
    z = np.zeros((2, 3, 4, 8))
    for fi, row in enumerate(frames):
        for p, key in enumerate(row):
            z[fi // 3, fi % 3, p, :2] = vec[key]
    cases = []
    for tau in (0.5, 0.6, 0.9, 0.96, 0.99):
        keep, sim, index = oracle.temporal_drop(z, tau)
        cases.append({"tau": tau, "keep": keep.astype(int).tolist(), "sim": sim.tolist(), "index": index.tolist()})
    return {"citation": "Sec. 3, Token Dropping (pairwise cosine over the chunk's frames, anchor frame)",
            "vectors": {k: list(v) for k, v in vec.items()}, "frames": frames, "dm": 8, "cases": cases}


def main():
    for fn, data in (("attention_uniform.json", attention_uniform_cases()), ("gather_uniform.json", gather_uniform_cases()),
                     ("acn_windows.json", acn_cases()),
                     ("drop_exact_cosines.json", drop_cases())):
        with open(os.path.join(HERE, fn), "w") as f:
            json.dump(data, f, indent=1)
            f.write("\n")


if __name__ == "__main__":
    main()
