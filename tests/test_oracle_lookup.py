"""Pins of the oracle's lookup and cache selector (Sec. 4.3 Alg. 1, Sec. 5.3.1).

The oracle is checked against things other than itself: exact rational
arithmetic, a literal per-element float64 loop, hand-built caches whose answer
is known, and the paper's selector table (tests/golden/selector_grid.txt).
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import lookup as LK

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
T_PAPER = [t for t, _ in synth.THRESHOLDS_PAPER]
K_PAPER = [k for _, k in synth.THRESHOLDS_PAPER]


def _rand_cache(n, d, seed, dtype):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, d)).astype(np.float32)
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    return synth.to_bf16_bits(x) if dtype == "bf16" else x


def _rows(cache):
    return synth.from_bf16_bits(cache) if cache.dtype == np.uint16 else cache


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_canonical_score_literal_loop_and_exact_bound(dtype):
    """(P-L1) float64 left-to-right scores: bit-equal to a literal Python loop and
    within d * 2^-53 * sum|q_k c_k| of the exact rational dot product."""
    cache = _rand_cache(48, 24, 7, dtype)
    q = _rand_cache(1, 24, 8, "f32")[0]
    got = LK.canonical_scores(q, cache)
    rows = _rows(cache)
    for i in range(cache.shape[0]):
        s = 0.0
        for k in range(24):
            s += float(q[k]) * float(rows[i, k])
        assert got[i] == s
        exact = sum(Fraction(float(q[k])) * Fraction(float(rows[i, k])) for k in range(24))
        bound = 24 * 2.0 ** -53 * sum(abs(float(q[k]) * float(rows[i, k])) for k in range(24))
        assert abs(Fraction(got[i]) - exact) <= Fraction(bound)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_top1_matches_exact_rational_argmax(dtype):
    """(P-L1) brute force: the selected index is the argmax of the exact dot products."""
    cache = _rand_cache(200, 16, 3, dtype)
    qs = _rand_cache(6, 16, 4, "f32")
    idx, sim, _ = LK.lookup(qs, cache, T_PAPER, K_PAPER)
    rows = _rows(cache)
    for j in range(qs.shape[0]):
        exact = [sum(Fraction(float(qs[j, k])) * Fraction(float(rows[i, k])) for k in range(16))
                 for i in range(rows.shape[0])]
        best = max(exact)
        assert idx[j] == exact.index(best)
        assert sim[j] == np.float32(float(best))


def test_ties_go_to_lowest_index():
    """(P-L2) exact duplicate rows i < j: the answer is i even when the query was built on j."""
    cache = _rand_cache(64, 32, 5, "bf16")
    cache[41] = cache[9]
    cache[60] = cache[9]
    tgt = synth.from_bf16_bits(cache[60:61])
    q = synth.make_queries_at_sims(tgt, [0.97], 1)
    idx, _, _ = LK.lookup(q, cache, T_PAPER, K_PAPER)
    assert idx[0] == 9
    assert LK.top1([1.0, 3.0, 2.0, 3.0]) == (1, 3.0)


def _one_hot_lookup(v):
    d = 8
    q = np.zeros((1, d), dtype=np.float32)
    q[0, 0] = 1.0
    cache = np.zeros((3, d), dtype=np.float32)
    cache[0, 1] = 1.0            # orthogonal row, score 0
    cache[1, 0] = np.float32(v)  # the match, score exactly v
    cache[2, 0] = -1.0
    return LK.lookup(q, cache, T_PAPER, K_PAPER)


@pytest.mark.parametrize("thr,k_at,k_above", [(0.95, 20, 25), (0.90, 15, 20), (0.85, 10, 15),
                                              (0.75, 5, 10), (0.65, 0, 5)])
def test_threshold_boundaries_through_lookup(thr, k_at, k_above):
    """(P-L3) a score exactly at a float32 threshold falls to the next K; one ulp above takes it."""
    t32 = np.float32(thr)
    idx, sim, kk = _one_hot_lookup(t32)
    assert idx[0] == 1 and sim[0] == t32 and kk[0] == k_at
    up = np.nextafter(t32, np.float32(2.0))
    idx, sim, kk = _one_hot_lookup(up)
    assert sim[0] == up and kk[0] == k_above


def test_selector_matches_paper_table():
    """(P-L4) the K map against the paper's table, read from the golden grid."""
    n = 0
    with open(os.path.join(GOLDEN, "selector_grid.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            s, k = line.split()
            assert LK.select_k(np.float32(float(s)), T_PAPER, K_PAPER) == int(k), s
            n += 1
    assert n >= 20


def test_empty_cache_and_negative_scores():
    """(P-L5) n = 0 gives (-1, -inf, 0); all-negative scores give K = 0 and the least
    negative row."""
    q = np.ones((2, 8), dtype=np.float32) / math.sqrt(8)
    idx, sim, kk = LK.lookup(q, np.zeros((0, 8), dtype=np.float32), T_PAPER, K_PAPER)
    assert list(idx) == [-1, -1] and np.all(np.isneginf(sim)) and list(kk) == [0, 0]
    cache = -np.abs(_rand_cache(30, 8, 2, "f32"))
    idx, sim, kk = LK.lookup(q, cache, T_PAPER, K_PAPER)
    ref = cache @ q[0]
    assert idx[0] == int(np.argmax(ref)) and sim[0] < 0 and kk[0] == 0


def test_synthetic_queries_hit_their_target_band():
    """Recipe check: a query built at similarity s to entry j scores s with j (float32 level)."""
    cache = synth.make_cache(1024, 64, 16, 0.1, 1, "f32")
    tg = [5, 100, 900]
    q = synth.make_queries_at_sims(cache[tg], [0.99, 0.93, 0.85], 2)
    for j, t in enumerate(tg):
        sc = LK.canonical_scores(q[j], cache)
        assert abs(sc[t] - [0.99, 0.93, 0.85][j]) < 1e-5
