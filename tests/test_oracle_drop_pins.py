"""Pins of the temporal token-dropping oracle (paper, Sec. 3, "Token
Dropping": pairwise cosine over all frame pairs of a chunk at each spatial
position, drop iff all exceed tau, first frame kept as anchor; c = 1 compares
with the previous frame and keeps no anchor)."""
from __future__ import annotations

import itertools

import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle
from oracle import token_drop as TD
from synth import make_drop_frames

f64 = oracle.bf16_bits_to_f64


def _brute(z, tau, prev=None):
    """Position by position with scipy's cosine distance and Python's all()."""
    B, c, n_f, _ = z.shape
    keep = np.ones((B, n_f), bool)
    for b in range(B):
        for p in range(n_f):
            if c > 1:
                s = 1.0 - cdist(z[b, :, p], z[b, :, p], metric="cosine")
                keep[b, p] = not all(s[i, j] > tau for i, j in itertools.combinations(range(c), 2))
            else:
                before = z[b - 1, 0, p] if b > 0 else (None if prev is None else prev[p])
                if before is not None:
                    s = 1.0 - cdist(z[b, 0, p][None], before[None], metric="cosine")[0, 0]
                    keep[b, p] = not s > tau
    index = [(b * c + f) * n_f + p for b in range(B) for f in range(c) for p in range(n_f)
             if (c > 1 and f == 0) or keep[b, p]]
    return keep, np.array(index)


@pytest.mark.parametrize("shape,tau", [((3, 4, 24, 64), 0.9), ((2, 2, 40, 128), 0.8), ((1, 8, 50, 256), 0.95),
                                       ((2, 3, 30, 32), 0.0)])
def test_matches_brute_force_with_scipy(shape, tau):
    z = f64(make_drop_frames(*shape, seed=sum(shape)))
    keep, sim, index = oracle.temporal_drop(z, tau)
    bk, bi = _brute(z, tau)
    assert np.array_equal(keep, bk) and np.array_equal(index, bi)
    # the reported similarity is the smallest pairwise cosine
    B, c, n_f, _ = z.shape
    for b in range(B):
        for p in range(0, n_f, 7):
            s = 1.0 - cdist(z[b, :, p], z[b, :, p], metric="cosine")
            assert abs(sim[b, p] - min(s[i, j] for i, j in itertools.combinations(range(c), 2))) <= 1e-12


def test_frame_level_chain_matches_brute_force():
    z = f64(make_drop_frames(6, 1, 32, 96, seed=3))
    prev = f64(make_drop_frames(1, 1, 32, 96, seed=4))[0, 0]
    for pv in (None, prev, z[0, 0]):
        keep, sim, index = oracle.temporal_drop(z, 0.7, prev=pv)
        bk, bi = _brute(z, 0.7, pv)
        assert np.array_equal(keep, bk) and np.array_equal(index, bi)
    keep, sim, _ = oracle.temporal_drop(z, 0.7)
    assert np.all(keep[0]) and np.all(sim[0] == oracle.NO_COMPARISON)      # nothing before the first frame
    keep, sim, _ = oracle.temporal_drop(z, 0.7, prev=z[0, 0])
    assert not np.any(keep[0])                                               # a frame equal to the previous one


def test_threshold_is_strict_at_an_exact_cosine():
    """(3, 4) and (4, 3) have cosine 24/25 exactly; tau = 0.96 does not drop."""
    z = np.zeros((1, 2, 1, 4))
    z[0, 0, 0, :2] = (3, 4)
    z[0, 1, 0, :2] = (4, 3)
    keep, sim, index = oracle.temporal_drop(z, 0.96)
    assert sim[0, 0] == 0.96 and keep[0, 0] and list(index) == [0, 1]
    keep, _, index = oracle.temporal_drop(z, 0.9599999)
    assert not keep[0, 0] and list(index) == [0]


def test_all_pairs_not_only_neighbours():
    """f1 = a, f2 = (a + b)/sqrt2, f3 = b with a orthogonal to b: neighbours have
    cosine 0.707 but frames 1 and 3 have 0, so tau = 0.5 keeps the position."""
    a, b = np.eye(3)[0], np.eye(3)[1]
    z = np.stack([a, (a + b) / np.sqrt(2), b])[None, :, None, :]
    keep, sim, _ = oracle.temporal_drop(z, 0.5)
    assert keep[0, 0] and abs(sim[0, 0]) <= 1e-15


def test_identical_frames_keep_only_the_anchor():
    z = np.repeat(f64(make_drop_frames(2, 1, 10, 16, seed=5)), 4, axis=1)     # [2, 4, 10, 16]
    keep, sim, index = oracle.temporal_drop(z, 0.5)
    assert not keep.any() and np.allclose(sim, 1.0, atol=1e-14)
    assert list(index) == [(b * 4) * 10 + p for b in range(2) for p in range(10)]
    tokens = oracle.gather_tokens(z, index)
    assert np.array_equal(tokens, z[:, 0].reshape(20, 16))


def test_unrelated_frames_keep_everything_in_stream_order():
    rng = np.random.default_rng(0)
    z = np.zeros((2, 3, 5, 16))
    for b in range(2):
        for f in range(3):
            z[b, f, :, 5 * f + b] = 1 + rng.random(5)         # disjoint supports: cosine 0
    keep, sim, index = oracle.temporal_drop(z, 0.1)
    assert keep.all() and np.all(sim == 0) and np.array_equal(index, np.arange(30))


def test_count_formula_and_order():
    z = f64(make_drop_frames(5, 4, 40, 32, seed=6))
    for tau in (0.5, 0.9, 0.97):
        keep, _, index = oracle.temporal_drop(z, tau)
        assert len(index) == sum(40 + 3 * int(k.sum()) for k in keep)
        assert np.all(np.diff(index) > 0)


def test_monotone_in_tau():
    z = f64(make_drop_frames(3, 4, 60, 48, seed=7))
    prev_keep = None
    for tau in np.linspace(-0.2, 1.0, 13):
        keep, _, _ = oracle.temporal_drop(z, tau)
        if prev_keep is not None:
            assert np.all(keep >= prev_keep)           # a higher threshold never drops more
        prev_keep = keep


def test_zero_vectors_have_cosine_zero():
    z = np.zeros((1, 3, 2, 8))
    z[0, :, 1, 0] = 1.0
    keep, sim, _ = oracle.temporal_drop(z, -0.5)
    assert np.all(sim[0] == [0.0, 1.0]) and not keep.any()
