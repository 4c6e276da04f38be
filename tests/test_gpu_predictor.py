"""GPU parity of the match predictor's gate (Sec. 5.2, Alg. 1): decision values
bit-exact against the oracle's left-to-right float64 scores, and the lookup
with the predictor in front equal to the oracle's: a predicted miss is
(-1, -inf, K = 0), every other query keeps its exact lookup result."""
import numpy as np
import pytest
import torch

import synth
from oracle import lookup as LK
from oracle import predictor as PR

pytestmark = pytest.mark.gpu

TP = [t for t, _ in synth.THRESHOLDS_PAPER]
KP = [k for _, k in synth.THRESHOLDS_PAPER]


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("d,n,m", [(768, 4000, 37), (64, 1000, 300), (8, 50, 5)])
def test_gate_scores_bit_exact(d, n, m):
    import paper_2312_04429_amd as P
    print(f"match gate scores d={d} n={n} m={m}", flush=True)
    X = synth.make_cache(n, d, 16, 0.1, 7, "bf16")
    rng = np.random.default_rng(d)
    w, rho = P.nv_ocsvm_train(X, 0.01, rng.integers(0, n, 4 * n))
    Q = np.concatenate([synth.from_bf16_bits(X[:m // 2]),
                        synth.make_prompt_stream(m - m // 2, d, 3, p_new=1.0)])
    got = P.nv_match_gate(t(Q), t(w), rho).cpu().numpy()
    want = PR.scores(w, rho, Q)
    assert np.array_equal(got, want)


def test_lookup_with_predictor_matches_oracle():
    """Alg. 1 with the predictor: near-duplicates of cached prompts and fresh draws;
    the threshold sits at a decision value so a query lands exactly on it."""
    import paper_2312_04429_amd as P
    n, d = 20000, 768
    X = synth.make_cache(n, d, 64, 0.05, 11, "bf16")
    rng = np.random.default_rng(5)
    w, rho = P.nv_ocsvm_train(X, 0.001, rng.integers(0, n, 3 * n))
    rows = synth.from_bf16_bits(X[rng.integers(0, n, 24)])
    near = synth.make_queries_at_sims(rows, rng.choice([0.97, 0.92, 0.87, 0.8, 0.7], 24), 6)
    fresh = synth.make_prompt_stream(24, d, 8, p_new=1.0)
    Q = np.concatenate([near, fresh])
    s = PR.scores(w, rho, Q)
    tau = float(np.sort(s)[len(s) // 2])
    print(f"predictor: {int((s >= tau).sum())} of {len(s)} predicted matches", flush=True)
    idx, sim, kk = P.nv_cache_lookup(t(Q), t(X.view(np.int16)), TP, KP)
    P.nv_match_gate(t(Q), t(w), rho, tau, idx, sim, kk, score=False)
    oi, osim, ok = LK.lookup(Q, X, TP, KP)
    keep = s >= tau
    oi, osim, ok = np.where(keep, oi, -1), np.where(keep, osim, -np.inf), np.where(keep, ok, 0)
    assert idx.cpu().numpy().tolist() == oi.tolist()
    assert kk.cpu().numpy().tolist() == ok.tolist()
    assert np.array_equal(sim.cpu().numpy(), osim.astype(np.float32))


def test_gated_lookup_searches_only_predicted_matches():
    """nv_cache_lookup_gated (the predictor in front of the search, Alg. 1):
    bit-exact against the oracle's lookup with predicted misses turned into
    (-1, -inf, K = 0); decision values bit-exact; the number searched equals
    the number predicted; and the two ends: tau above every score (nothing
    searched) and below every score (the plain lookup's result).  Both cache
    types hold the same values (bf16 rows widened to float32), so one oracle
    result serves both."""
    import paper_2312_04429_amd as P
    n, d, m = 6000, 768, 160
    X = synth.make_cache(n, d, 64, 0.05, 13, "bf16")
    rng = np.random.default_rng(9)
    w, rho = P.nv_ocsvm_train(X, 0.001, rng.integers(0, n, 3 * n))
    Xf = synth.from_bf16_bits(X)
    rows = Xf[rng.integers(0, n, m // 2)]
    near = synth.make_queries_at_sims(rows, rng.choice([0.97, 0.92, 0.87, 0.8, 0.7], m // 2), 3)
    fresh = synth.make_prompt_stream(m // 2, d, 4, p_new=1.0)
    Q = np.concatenate([near, fresh])[rng.permutation(m)]
    s = PR.scores(w, rho, Q)
    oi, osim, ok = LK.lookup(Q, X, TP, KP)
    for name, cache in (("bf16", t(X.view(np.int16))), ("f32", t(Xf))):
        for tau in (float(np.sort(s)[m // 3]), float(s.max()) + 1.0, float(s.min()) - 1.0):
            keep = s >= tau
            print(f"gated lookup {name} tau={tau:.4g}: {int(keep.sum())} of {m}", flush=True)
            idx, sim, kk, score, searched = P.nv_cache_lookup_gated(t(Q), cache, TP, KP, t(w),
                                                                    rho, tau)
            assert searched == int(keep.sum())
            assert np.array_equal(score.cpu().numpy(), s)
            assert idx.cpu().numpy().tolist() == np.where(keep, oi, -1).tolist()
            assert kk.cpu().numpy().tolist() == np.where(keep, ok, 0).tolist()
            assert np.array_equal(sim.cpu().numpy(),
                                  np.where(keep, osim, -np.inf).astype(np.float32))
