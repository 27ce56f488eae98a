"""Log-sum-exp merge of attention computed over disjoint key sets (oracle side).

If the visible keys of a row are split into disjoint parts s with partial
results (O_s, lse_s) -- each O_s the softmax-weighted average over its part
and lse_s the natural-log normaliser of that part -- then the whole-set
result is lse = log(sum_s exp(lse_s)) and O = sum_s exp(lse_s - lse) O_s.
This is the identity exp(z_j - lse) = exp(lse_s - lse) * exp(z_j - lse_s)
summed over each part.  It is used to pin the split-key-range path of the
library.  Parts with no visible key carry lse_s = -inf and contribute 0.
Test infrastructure only.
"""
from __future__ import annotations

import numpy as np


def lse_merge(outs, lses):
    """outs: list of [..., dv] arrays; lses: list of [...] arrays (natural log)."""
    L = np.stack([np.asarray(x, dtype=np.float64) for x in lses])       # [P, ...]
    O = np.stack([np.asarray(x, dtype=np.float64) for x in outs])       # [P, ..., dv]
    m = np.max(L, axis=0)
    m_safe = np.where(np.isfinite(m), m, 0.0)
    w = np.exp(L - m_safe)                                               # exp(-inf) = 0
    tot = np.sum(w, axis=0)
    with np.errstate(divide="ignore", invalid="ignore"):
        lse = np.where(tot > 0, m_safe + np.log(np.where(tot > 0, tot, 1.0)), -np.inf)
        wn = np.where(tot > 0, w / np.where(tot > 0, tot, 1.0), 0.0)
    O = np.where(np.isfinite(O), O, 0.0)
    out = np.sum(wn[..., None] * O, axis=0)
    return out, lse
