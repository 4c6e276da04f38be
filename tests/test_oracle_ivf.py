"""Pins of the oracle's IVF index (approximate search over the vector DB,
Sec. 5.3 / Sec. 6: the paper's vector DB searches through an index).

Checked against things other than itself: probing every list (or a single
list) reduces to the exact lookup, which has its own pins; a hand-built circle
of embeddings whose lists and probe results are worked out by hand; the
normalised-mean update against an independent numpy mean; the spherical
k-means objective never decreasing over Lloyd steps (float32 cache); list
bookkeeping against brute force; and monotonicity of the result in nprobe.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import ivf
from oracle import lookup as LK

T = [t for t, _ in synth.THRESHOLDS_PAPER]
K = [k for _, k in synth.THRESHOLDS_PAPER]


def _queries(X, m, seed):
    rows = synth.from_bf16_bits(X) if X.dtype == np.uint16 else X
    rng = np.random.default_rng(seed)
    near = synth.make_queries_at_sims(rows[rng.integers(0, len(rows), m // 2)],
                                      rng.choice([0.97, 0.9, 0.8, 0.7], m // 2), seed)
    return np.concatenate([near, synth.make_prompt_stream(m - m // 2, X.shape[1], seed,
                                                          p_new=1.0)])


@pytest.mark.parametrize("dtype,L,iters", [("bf16", 12, 0), ("bf16", 8, 2), ("f32", 5, 1)])
def test_probing_all_lists_is_the_exact_lookup(dtype, L, iters):
    X = synth.make_cache(600, 32, 6, 0.15, 3, dtype, dup_pairs=((5, 17), (40, 41)))
    init = np.random.default_rng(L).choice(600, L, replace=False)
    c, lists, perm, off = ivf.build(X, init, iters)
    q = _queries(X, 16, 4)
    q[0] = synth.from_bf16_bits(X[5]) if dtype == "bf16" else X[5]     # exact duplicate rows
    for nprobe in (L,):
        i1, s1, k1, _ = ivf.search(q, X, c, perm, off, nprobe, T, K)
        i2, s2, k2 = LK.lookup(q, X, T, K)
        assert i1.tolist() == i2.tolist() and k1.tolist() == k2.tolist()
        assert np.array_equal(s1, s2)
    assert i1[0] == 5                                   # tie between rows 5 and 17 -> 5
    c1, _, p1, o1 = ivf.build(X, init[:1], 0)
    i3, s3, k3, _ = ivf.search(q, X, c1, p1, o1, 1, T, K)
    assert i3.tolist() == i2.tolist() and np.array_equal(s3, s2)


def test_circle_by_hand():
    """Unit vectors at 0, 85, 180, 170 degrees; centroids rows 0 and 2 give lists
    {0, 1} (85 is nearer 0 than 180) and {2, 3}.  A query at 92 degrees scores
    cos 92 < 0 < cos 88 against the centroids, so list 1 is probed first: with one
    probe the answer is row 3 (cos 78), although row 1 (cos 7) is the nearest row;
    with two probes it is row 1."""
    ang = np.radians([0, 85, 180, 170])
    X = np.stack([np.cos(ang), np.sin(ang)], 1).astype(np.float32)
    c, lists, perm, off = ivf.build(X, [0, 2], 0)
    assert lists.tolist() == [0, 0, 1, 1] and off.tolist() == [0, 2, 4]
    q = np.array([[math.cos(math.radians(92)), math.sin(math.radians(92))]], np.float32)
    i1, s1, _, pr = ivf.search(q, X, c, perm, off, 1, T, K)
    assert pr.tolist() == [[1]] and i1.tolist() == [3]
    assert abs(s1[0] - math.cos(math.radians(78))) < 1e-6
    i2, s2, _, pr = ivf.search(q, X, c, perm, off, 2, T, K)
    assert pr.tolist() == [[1, 0]] and i2.tolist() == [1]
    assert abs(s2[0] - math.cos(math.radians(7))) < 1e-6


def test_lloyd_update_is_the_normalised_mean():
    X = synth.make_cache(300, 16, 3, 0.2, 9, "f32")
    init = [0, 100, 200]
    c0 = X[init].copy()
    lists = ivf.assign(X, c0)
    c1 = ivf.lloyd_centroids(X, lists, c0)
    for l in range(3):
        mu = X[lists == l].astype(np.float64).mean(0)
        np.testing.assert_allclose(c1[l], mu / np.linalg.norm(mu), rtol=2e-7, atol=1e-8)


def test_lloyd_never_lowers_the_objective():
    X = synth.make_cache(800, 24, 8, 0.2, 11, "f32")
    init = np.random.default_rng(1).choice(800, 10, replace=False)
    c = X[init].copy()
    prev = -np.inf
    for _ in range(5):
        lists = ivf.assign(X, c)
        obj = float(sum(X[i].astype(np.float64) @ c[lists[i]].astype(np.float64)
                        for i in range(800)))
        assert obj >= prev - 1e-6 * abs(obj)
        prev = obj
        c = ivf.lloyd_centroids(X, lists, c)


def test_lists_against_brute_force_and_nprobe_monotone():
    X = synth.make_cache(500, 16, 5, 0.2, 13, "bf16")
    init = np.random.default_rng(2).choice(500, 9, replace=False)
    c, lists, perm, off = ivf.build(X, init, 1)
    rows = synth.from_bf16_bits(X).astype(np.float64)
    cf = synth.from_bf16_bits(c).astype(np.float64)
    sc = rows @ cf.T
    best = sc.max(1)
    for i in range(500):                 # chosen list is a maximiser (float64 matmul agrees)
        assert sc[i, lists[i]] >= best[i] - 1e-12
    assert sorted(perm.tolist()) == list(range(500))
    for l in range(9):
        seg = perm[off[l]:off[l + 1]]
        assert (np.diff(seg) > 0).all() and (lists[seg] == l).all()
    q = _queries(X, 12, 5)
    prev = None
    for nprobe in range(1, 10):
        _, s, _, _ = ivf.search(q, X, c, perm, off, nprobe, T, K)
        if prev is not None:
            assert (s >= prev).all()
        prev = s


def test_duplicate_centroids_ties_and_empty_lists():
    """Rows 7 and 8 are identical and both start a centroid: every row scores them
    equally, so the lower list takes all of them and list 1 stays empty; a query's tie
    between the two goes to the lower list, so one probe finds row 7 itself.  Through a
    Lloyd step the empty list keeps its centroid."""
    X = synth.make_cache(200, 16, 4, 0.2, 21, "bf16", dup_pairs=((7, 8),))
    c, lists, perm, off = ivf.build(X, [7, 8, 50, 120], 0)
    assert off[2] - off[1] == 0 and (lists != 1).all()
    q = synth.from_bf16_bits(X[7:8])
    i1, _, _, pr = ivf.search(q, X, c, perm, off, 1, T, K)
    assert pr[0, 0] == 0 and i1[0] == 7
    c1, _, _, _ = ivf.build(X, [7, 8, 50, 120], 1)
    assert np.array_equal(c1[1], X[8])


def test_round_like_matches_torch_rounding():
    """The centroid storage rounding (float64 -> float32 -> bfloat16, nearest
    even at each step) against torch's own conversions, on values built to sit
    exactly on and one ulp either side of bfloat16 ties (both parities of the
    kept bit), at both signs, in the subnormal range and next to the largest
    finite bfloat16.  A truncating or ties-away rounding fails here."""
    rng = np.random.default_rng(5)
    hi = rng.integers(0, 0x7F7F, 4000, dtype=np.uint32)  # finite bf16 patterns below the max
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF], np.uint32)
    u = (hi[:, None] << np.uint32(16)) | lows[None, :]
    f32 = u.reshape(-1).view(np.float32)
    vals = np.concatenate([f32, -f32]).astype(np.float64)
    # float64 values between float32 neighbours (the first rounding matters too)
    vals = np.concatenate([vals, vals * (1 + 2.0 ** -30), rng.standard_normal(4000) * 1e-39,
                           np.array([3.3895313892515355e38, -3.3895313892515355e38])])
    got = ivf._round_like(vals, np.uint16)
    ref = torch.tensor(vals, dtype=torch.float64).to(torch.float32).to(torch.bfloat16)
    np.testing.assert_array_equal(got, ref.view(torch.int16).numpy().view(np.uint16))
    np.testing.assert_array_equal(ivf._round_like(vals, np.float32),
                                  torch.tensor(vals).to(torch.float32).numpy())
