"""GPU parity of the cache lookup and state fetch against the oracle.

Bar: idx, sim and K bit-identical to the oracle (Sec. 4.3 Alg. 1 search +
Sec. 5.3.1 selector), at small sizes spanning several 128- and 256-row tiles
with ragged tails and several 16-query blocks, on the edge cases (ties,
overflowing candidate lists, empty cache, threshold boundaries) and at the
workloads' full sizes (exact for sampled queries, properties for the rest).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import lookup as LK

pytestmark = pytest.mark.gpu

TP = [t for t, _ in synth.THRESHOLDS_PAPER]
KP = [k for _, k in synth.THRESHOLDS_PAPER]


def _gpu_lookup(q, cache, thr=TP, kv=KP):
    import paper_2312_04429_amd as P
    qd = torch.from_numpy(np.ascontiguousarray(q)).cuda()
    if cache.dtype == np.uint16:
        cd = torch.from_numpy(cache.view(np.int16)).cuda() if cache.size else \
            torch.empty((0, cache.shape[1]), dtype=torch.int16, device="cuda")
    else:
        cd = torch.from_numpy(np.ascontiguousarray(cache)).cuda()
    idx, sim, kk = P.nv_cache_lookup(qd, cd, thr, kv)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), sim.cpu().numpy(), kk.cpu().numpy()


def _check(q, cache, thr=TP, kv=KP):
    gi, gs, gk = _gpu_lookup(q, cache, thr, kv)
    oi, os_, ok = LK.lookup(q, cache, thr, kv)
    np.testing.assert_array_equal(gi, oi)
    np.testing.assert_array_equal(gs.view(np.uint32), os_.view(np.uint32))
    np.testing.assert_array_equal(gk, ok)
    return gi, gs, gk


def _rand(n, d, seed, dtype):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, d)).astype(np.float32)
    x /= np.linalg.norm(x, axis=1, keepdims=True) + 1e-30
    return synth.to_bf16_bits(x) if dtype == "bf16" else x


def test_tiny_workload():
    w = synth.WORKLOADS["tiny"]
    print("lookup tiny workload", flush=True)
    cache = synth.make_cache(w["n_cache"], w["d"], w["clusters"], w["sigma"], w["cache_seed"],
                             "f32", dup_pairs=((300, 700),))
    tg = [700, 5, 100, 900, 512, 40]
    q = synth.make_queries_at_sims(cache[tg], w["query_sims"], w["query_seed"])
    q2 = synth.make_cluster_queries(w["n_cluster_queries"], w["d"], w["clusters"], w["sigma"],
                                    w["cache_seed"], w["query_seed"])
    q = np.concatenate([q, q2])
    thr = [t for t, _ in w["thresholds"]]
    kv = [k for _, k in w["thresholds"]]
    gi, _, gk = _check(q, cache, thr, kv)
    assert gi[0] == 300                      # duplicate rows: lowest index
    assert list(gk[:2]) == [10, 10]


@pytest.mark.parametrize("n,d,m", [(1, 64, 1), (255, 64, 3), (257, 768, 8), (5000, 768, 17),
                                   (1500, 40, 40), (777, 2048, 2), (129, 768, 33),
                                   (300, 1024, 20)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_random_caches(n, d, m, dtype):
    print(f"lookup random n={n} d={d} m={m} {dtype}", flush=True)
    cache = _rand(n, d, n + d, dtype)
    rows = synth.cache_rows_f32(cache, np.arange(min(n, m)) * 7 % n)
    q = np.concatenate([synth.make_queries_at_sims(rows, np.linspace(0.99, 0.6, len(rows)), 3),
                        _rand(max(0, m - len(rows)), d, 9, "f32")])
    _check(q, cache)


def test_overflowing_candidate_lists():
    """200 identical rows inside one tile and whole tiles of identical rows."""
    print("lookup overflow", flush=True)
    cache = _rand(4000, 768, 1, "bf16")
    cache[50:250] = cache[1234]
    q = synth.make_queries_at_sims(synth.cache_rows_f32(cache, [1234]), [0.97], 4)
    gi, _, gk = _check(q, cache)
    assert gi[0] == 50 and gk[0] == 25
    # the same cache with 20 queries (two query blocks), all near the duplicated row
    q20 = synth.make_queries_at_sims(synth.cache_rows_f32(cache, [1234] * 20),
                                     np.linspace(0.99, 0.9, 20), 6)
    gi, _, _ = _check(q20, cache)
    assert np.all(gi == 50)
    same = np.repeat(_rand(1, 64, 2, "bf16"), 700 * 256 + 3, axis=0)  # > 512 overflowing tiles
    q = synth.make_queries_at_sims(synth.cache_rows_f32(same, [0]), [0.9], 5)
    gi, _, _ = _check(q, same)
    assert gi[0] == 0


@pytest.mark.parametrize("d,dtype", [(768, "bf16"), (64, "bf16"), (1024, "bf16"), (768, "f32")])
def test_scan_rounding_inversion(d, dtype):
    """The bf16 scan orders two rows the wrong way round; the margins must keep
    the true best.  Row 0 = 1.0 e_2 scores q_2 = 1.0038 canonically but 1.0 in
    the scan (q_2 rounds down to bf16 1.0); row 300 = 0.70703125 (e_3 + e_4)
    scores 1.0030 canonically but 1.0053 in the scan (q_3 = q_4 = 0.7093 round
    up to 0.7109375).  The nonzeros sit at k % 8 in 2..4, so a row-norm bound
    that read only part of each 8-element chunk would be 0 and the row-0 tile
    would be dropped.  Every other row is zero."""
    print(f"lookup rounding inversion d={d} {dtype}", flush=True)
    q = np.zeros((1, d), dtype=np.float32)
    q[0, 2], q[0, 3], q[0, 4] = 1.0038, 0.7093, 0.7093
    c = np.zeros((400, d), dtype=np.float32)
    c[0, 2] = 1.0
    c[300, 3] = c[300, 4] = 0.70703125
    cache = synth.to_bf16_bits(c) if dtype == "bf16" else c
    gi, gs, gk = _check(q, cache)
    assert gi[0] == 0 and gk[0] == 25
    # the same pair in a cache of unit rows, several queries (m > 1 query block)
    rng = _rand(4000, d, 17, "f32") * 0.2
    rng[0], rng[3000] = c[0], c[300]
    cache = synth.to_bf16_bits(rng) if dtype == "bf16" else rng
    gi, _, _ = _check(np.repeat(q, 20, axis=0), cache)
    assert np.all(gi == 0)


def test_empty_cache_and_boundaries():
    print("lookup empty + boundaries", flush=True)
    q = _rand(3, 64, 1, "f32")
    gi, gs, gk = _gpu_lookup(q, np.zeros((0, 64), dtype=np.float32))
    assert list(gi) == [-1] * 3 and np.all(np.isneginf(gs)) and list(gk) == [0] * 3
    gi, gs, gk = _gpu_lookup(q, np.zeros((0, 64), dtype=np.uint16))
    assert list(gi) == [-1] * 3
    # one-hot queries against rows scoring exactly at / one ulp above each threshold
    vals = []
    for t in TP:
        t32 = np.float32(t)
        vals += [t32, np.nextafter(t32, np.float32(2))]
    d = 64
    cache = np.zeros((len(vals), d), dtype=np.float32)
    q = np.zeros((len(vals), d), dtype=np.float32)
    for i, v in enumerate(vals):
        cache[i, i] = v
        q[i, i] = 1.0
    gi, gs, gk = _check(q, cache)
    assert list(gk) == [20, 25, 15, 20, 10, 15, 5, 10, 0, 5]


def test_sd15_b1_cache_full_size():
    w = synth.WORKLOADS["sd15_b1"]
    print("lookup 100k x 768 bf16", flush=True)
    cache = synth.make_cache(w["n_cache"], w["d"], w["clusters"], w["sigma"], w["cache_seed"])
    q = synth.make_queries_at_sims(synth.cache_rows_f32(cache, [31337]), w["query_sims"],
                                   w["query_seed"])
    gi, _, gk = _check(q, cache)
    assert gi[0] == 31337 and gk[0] == 25


def test_sd15_b8_cache_full_size_sampled():
    """1M x 768 bf16 with 8 queries (launch configuration of the benchmark); the oracle
    scores every row canonically for each query."""
    w = synth.WORKLOADS["sd15_b8_mixed"]
    print("lookup 1M x 768 bf16, 8 queries", flush=True)
    cache = synth.make_cache(w["n_cache"], w["d"], w["clusters"], w["sigma"], w["cache_seed"])
    tg = np.arange(8) * 123457 % w["n_cache"]
    sims = [0.97, 0.92, 0.87, 0.8, 0.7, 0.6, 0.99, 0.95]
    q = synth.make_queries_at_sims(synth.cache_rows_f32(cache, tg), sims, w["query_seed"])
    gi, gs, gk = _gpu_lookup(q, cache)
    for j in range(8):
        sc = LK.canonical_scores(q[j], cache)
        i, v = LK.top1_fast(sc)
        assert gi[j] == i and gs[j] == np.float32(v)
        assert gk[j] == LK.select_k(np.float32(v), TP, KP)
        print(f"  q{j}: idx {i} sim {v:.6f} K {gk[j]}", flush=True)


def test_256_queries_against_oracle():
    """The retrieval-heavy query shape (256 queries, half within cosine 0.95 of a cached
    row) on a 20k-row cache the oracle scans whole."""
    print("lookup 20k x 768 bf16, 256 queries", flush=True)
    cache = synth.make_cache(20_000, 768, 100, 0.05, 41)
    rng = np.random.default_rng(42)
    near = synth.make_queries_at_sims(synth.cache_rows_f32(cache, rng.choice(20_000, 128)),
                                      rng.uniform(0.95, 0.995, 128), 43)
    far = synth.make_cluster_queries(128, 768, 100, 0.05, 41, 44)
    gi, _, gk = _check(np.concatenate([near, far]), cache)
    assert np.all(gk[:128] >= 20)


def test_retrieval_heavy_full_size_sampled():
    """10M x 768 bf16 cache drawn on the device, 256 queries.  Exact against the oracle
    for one query (every row rescored canonically); for all 256: the returned row's
    canonical score gives sim and K, it dominates the planted row and a row sample."""
    import paper_2312_04429_amd as P
    w = synth.WORKLOADS["retrieval_heavy"]
    n, d = w["n_cache"], w["d"]
    print("lookup retrieval-heavy: drawing 10M x 768 on the device", flush=True)
    cache = synth.make_cache_device(n, d, w["clusters"], w["sigma"], w["cache_seed"], "cuda")
    mu = synth.cluster_centres_device(w["clusters"], d, w["cache_seed"], "cuda").cpu().numpy()
    rng = np.random.default_rng(w["query_seed"])
    half = w["n_queries"] // 2
    planted = rng.choice(n, half, replace=False)
    rows = cache[torch.from_numpy(planted).cuda()].view(torch.int16).cpu().numpy().view(np.uint16)
    near = synth.make_queries_at_sims(synth.from_bf16_bits(rows), rng.uniform(0.95, 0.995, half),
                                      w["query_seed"])
    far = synth.cluster_queries_from(mu, half, w["sigma"], w["query_seed"] + 1)
    q = np.concatenate([near, far])
    print("  lookup 256 queries", flush=True)
    idx, sim, kk = P.nv_cache_lookup(torch.from_numpy(q).cuda(), cache, TP, KP)
    gi, gs, gk = idx.cpu().numpy(), sim.cpu().numpy(), kk.cpu().numpy()

    def host_rows(r):
        t = cache[torch.from_numpy(np.asarray(r, dtype=np.int64)).cuda()]
        return t.view(torch.int16).cpu().numpy().view(np.uint16)

    best = host_rows(gi)
    sample = rng.choice(n, 4096, replace=False)
    samp = host_rows(sample)
    print("  properties for 256 queries", flush=True)
    for j in range(len(q)):
        sj = LK.canonical_scores(q[j], best[j:j + 1])[0]
        assert gs[j] == np.float32(sj) and gk[j] == LK.select_k(np.float32(sj), TP, KP)
        if j < half:
            sp = LK.canonical_scores(q[j], rows[j:j + 1])[0]
            assert sj > sp or (sj == sp and gi[j] <= planted[j])
        ss = LK.canonical_scores(q[j], samp)
        assert np.all((ss < sj) | ((ss == sj) & (sample >= gi[j])))
    assert np.all(gk[:half] >= 20)
    j = half  # a far query: every row through the oracle, 1M rows at a time
    print("  exact scan of one query over 10M rows (oracle)", flush=True)
    bi, bs = -1, -np.inf
    for start in range(0, n, 1 << 20):
        blk = cache[start:start + (1 << 20)].view(torch.int16).cpu().numpy().view(np.uint16)
        i, v = LK.top1_fast(LK.canonical_scores(q[j], blk))
        if v > bs:
            bi, bs = start + i, v
    print(f"  q{j}: oracle idx {bi} sim {bs:.6f}; gpu idx {gi[j]} sim {gs[j]:.6f}", flush=True)
    assert gi[j] == bi and gs[j] == np.float32(bs)


def test_gather_states():
    import paper_2312_04429_amd as P
    print("gather states", flush=True)
    rng = np.random.default_rng(0)
    n_store, slots, lat = 6, [5, 10, 15, 20, 25], (4, 8, 8)
    store = rng.standard_normal((n_store, len(slots)) + lat).astype(np.float32)
    noise = rng.standard_normal((5,) + lat).astype(np.float32)
    payload = np.array([3, 1, 5, 0, -1, 2, 4, 7], dtype=np.int32)  # row -> store entry
    idx = np.array([0, 2, 4, 1, 7], dtype=np.int64)
    kk = np.array([10, 25, 5, 0, 5], dtype=np.int32)
    t = lambda a: torch.from_numpy(a).cuda()
    kd = t(kk.copy())
    out = P.nv_gather_states(t(store), slots, t(payload), 8, t(idx), kd, t(noise)).cpu().numpy()
    kout = kd.cpu().numpy()
    np.testing.assert_array_equal(out[0], store[3, 1])
    np.testing.assert_array_equal(out[1], store[5, 4])
    np.testing.assert_array_equal(out[2], noise[2])   # payload -1: miss
    np.testing.assert_array_equal(out[3], noise[3])   # K = 0
    np.testing.assert_array_equal(out[4], noise[4])   # payload 7 out of range
    assert list(kout) == [10, 25, 0, 0, 0]
