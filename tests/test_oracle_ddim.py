"""Pins of the oracle's schedule, DDIM update, guidance and cache resumption.

Closed forms (Sec. 2.1 schedule, DDIM of Sec. 6) and the invariants of
approximate caching (Sec. 4.1): resuming from the state after K steps of a
full run reproduces that run's tail; K = 0 is the full run; K = N returns the
cached state unchanged (pure retrieval, Sec. 5.3.1).
"""
import math

import numpy as np
import pytest

import synth
from oracle import ddim, schedule
from oracle import unet as U

S = synth.SCHEDULE_SD


def test_beta_endpoints_and_alpha_product():
    b = schedule.betas(1000, 0.00085, 0.012)
    assert b[0] == pytest.approx(0.00085, rel=1e-12)
    assert b[-1] == pytest.approx(0.012, rel=1e-12)
    ac = schedule.alphas_cumprod64(1000, 0.00085, 0.012)
    # independent route: exp of a correctly rounded sum of logs
    for t in (0, 1, 480, 481, 880, 999):
        ref = math.exp(math.fsum(math.log1p(-float(x)) for x in b[:t + 1]))
        assert ac[t] == pytest.approx(ref, rel=1e-12)
    # decreasing, inside (0, 1)
    assert np.all(np.diff(ac) < 0) and 0 < ac[-1] < ac[0] < 1


def test_timestep_grid():
    ts = schedule.timesteps(50, 1000)
    assert ts[0] == 981 and ts[-1] == 1 and len(ts) == 50
    assert all(a - b == 20 for a, b in zip(ts, ts[1:]))
    ts = schedule.timesteps(20, 1000)
    assert ts[0] == 951 and ts[-1] == 1
    with pytest.raises(ValueError):
        schedule.timesteps(30, 1000)
    _, _, last_prev = schedule.step_alphas(49, 50, S)
    assert last_prev == schedule.alphas_cumprod(1000, 0.00085, 0.012)[0]


def test_alpha_values_at_skip_points():
    ac = schedule.alphas_cumprod(1000, 0.00085, 0.012)
    assert ac[981] == pytest.approx(0.005776, abs=2e-6)
    assert ac[481] == pytest.approx(0.302296, abs=2e-6)
    assert ac[0] == pytest.approx(0.99915, abs=1e-7)


def test_ddim_step_closed_forms():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(64).astype(np.float32)
    eps = rng.standard_normal(64).astype(np.float32)
    a_t, a_p = np.float32(0.3), np.float32(0.6)
    y = ddim.ddim_step(x, eps, a_t, a_p)
    x0 = (x.astype(np.float64) - math.sqrt(1 - 0.3) * eps) / math.sqrt(0.3)
    ref = math.sqrt(0.6) * x0 + math.sqrt(1 - 0.6) * eps
    np.testing.assert_allclose(y, ref, rtol=2e-6, atol=2e-6)
    # zero noise prediction scales by sqrt(a_p / a_t)
    np.testing.assert_allclose(ddim.ddim_step(x, 0 * eps, a_t, a_p), x * math.sqrt(0.6 / 0.3),
                               rtol=1e-6)
    # guidance
    eu, ec = x, eps
    np.testing.assert_allclose(ddim.cfg_combine(eu, ec, 7.5), eu + 7.5 * (ec - eu), rtol=1e-6)


def _tiny():
    cfg = synth.unet_config("tiny")
    w = synth.make_weights(cfg, 0)
    ctx = synth.make_contexts(2, cfg["ctx_len"], cfg["ctx_dim"], 3)
    x = synth.make_latents(1, 4, cfg["H"], cfg["W"], 2000)[0]
    return cfg, w, ctx, x


@pytest.mark.parametrize("K", [0, 5, 10])
def test_zero_eps_telescopes(K):
    """(C-P1) with conv_out zeroed eps = 0 and x_end = x_K sqrt(abar_end / abar_tK)."""
    cfg, w, ctx, x = _tiny()
    w = dict(w)
    w["conv_out.w"] = np.zeros_like(w["conv_out.w"])
    w["conv_out.b"] = np.zeros_like(w["conv_out.b"])
    net = U.UNet(cfg, w)
    out = ddim.denoise(U.make_eps_fn(net, ctx[0], ctx[1]), x, K, 20, S, 7.5)
    ac = schedule.alphas_cumprod64(1000, 0.00085, 0.012)
    tk = schedule.timesteps(20, 1000)[K]
    np.testing.assert_allclose(out, x * math.sqrt(ac[0] / ac[tk]), rtol=2e-5)


def test_constant_eps_closed_form():
    """(C-P2) conv_out weight 0 and bias b make eps = b for every row, so
    x_end / sqrt(abar_end) = x_K / sqrt(abar_tK) + b (sig_end - sig_tK), sig = sqrt((1-a)/a)."""
    cfg, w, ctx, x = _tiny()
    w = dict(w)
    b = np.array([0.3, -0.2, 0.1, 0.05], dtype=np.float32)
    w["conv_out.w"] = np.zeros_like(w["conv_out.w"])
    w["conv_out.b"] = b
    net = U.UNet(cfg, w)
    K = 5
    out = ddim.denoise(U.make_eps_fn(net, ctx[0], ctx[1]), x, K, 20, S, 7.5)
    ac = schedule.alphas_cumprod(1000, 0.00085, 0.012).astype(np.float64)
    tk = schedule.timesteps(20, 1000)[K]
    sig = lambda a: math.sqrt((1 - a) / a)
    ref = math.sqrt(ac[0]) * (x / math.sqrt(ac[tk]) + b[:, None, None] * (sig(ac[0]) - sig(ac[tk])))
    np.testing.assert_allclose(out, ref, rtol=1e-4, atol=1e-5)


def test_cfg_degenerate_and_resume_invariants():
    """(C-P3) cond == uncond makes the guidance scale irrelevant; (C-P4) resuming from the
    state after K steps reproduces the full run bitwise; (C-P5) K = N is the identity."""
    cfg, w, ctx, x = _tiny()
    net = U.UNet(cfg, w)
    same = U.make_eps_fn(net, ctx[0], ctx[0])
    a = ddim.denoise(same, x, 12, 20, S, 7.5)
    b = ddim.denoise(same, x, 12, 20, S, 1.0)
    np.testing.assert_array_equal(a, b)
    fn = U.make_eps_fn(net, ctx[0], ctx[1])
    states = {}
    full = ddim.denoise(fn, x, 0, 20, S, 7.5, record=lambda i, v: states.__setitem__(i, v))
    for K in (5, 10, 15):
        np.testing.assert_array_equal(ddim.denoise(fn, states[K], K, 20, S, 7.5), full)
    np.testing.assert_array_equal(ddim.denoise(fn, states[20], 20, 20, S, 7.5), states[20])
    np.testing.assert_array_equal(states[20], full)
    with pytest.raises(ValueError):
        ddim.denoise(fn, x, 21, 20, S, 7.5)


def test_guidance_one_is_conditional_only():
    cfg, w, ctx, x = _tiny()
    net = U.UNet(cfg, w)
    a = ddim.denoise(U.make_eps_fn(net, ctx[0], ctx[1]), x, 15, 20, S, 1.0)
    b = ddim.denoise(lambda v, t: (net(v, t, ctx[0]), net(v, t, ctx[0])), x, 15, 20, S, 1.0)
    np.testing.assert_allclose(a, b, rtol=1e-4, atol=1e-5)


@pytest.mark.parametrize("i", [0, 10, 24, 49])
def test_stochastic_step_eta0_and_eta1(i):
    """eta = 0 is the deterministic update bit for bit (any z).  eta = 1 matches the
    forward process's posterior q(x_prev | x_t, x_0) obtained by Gaussian conditioning
    (Schur complement of the joint of x_prev and x_t given x_0): variance and mean."""
    S = synth.SCHEDULE_SD
    _, a_t, a_p = schedule.step_alphas(i, 50, S)
    rng = np.random.default_rng(i)
    x0 = rng.standard_normal(64).astype(np.float32)
    e = rng.standard_normal(64).astype(np.float32)
    xt = (np.sqrt(np.float32(a_t)) * x0 + np.sqrt(np.float32(1 - a_t)) * e).astype(np.float32)
    z = rng.standard_normal(64).astype(np.float32)
    assert np.array_equal(ddim.ddim_step_eta(xt, e, a_t, a_p, 0.0, z), ddim.ddim_step(xt, e, a_t, a_p))
    at, ap = float(a_t), float(a_p)
    cov = math.sqrt(at / ap) * (1 - ap)                 # Cov(x_prev, x_t | x_0)
    var_post = (1 - ap) - cov * cov / (1 - at)
    sig = float(ddim.ddim_sigma(a_t, a_p, 1.0))
    assert abs(sig * sig - var_post) <= 1e-4 * var_post   # float32 sigma
    mean_post = math.sqrt(ap) * x0.astype(np.float64) + cov / (1 - at) * (
        xt.astype(np.float64) - math.sqrt(at) * x0)
    got = ddim.ddim_step_eta(xt, e, a_t, a_p, 1.0, np.zeros(64, np.float32))
    np.testing.assert_allclose(got, mean_post, rtol=0, atol=2e-5)


@pytest.mark.parametrize("eta", [0.0, 0.5, 1.0])
def test_stochastic_step_keeps_the_marginal(eta):
    """With the true eps, every member of the family maps x_t ~ q(x_t | x_0) to
    x_prev ~ q(x_prev | x_0): mean sqrt(a_prev) x_0, variance 1 - a_prev."""
    S = synth.SCHEDULE_SD
    _, a_t, a_p = schedule.step_alphas(20, 50, S)
    rng = np.random.default_rng(7)
    n = 400_000
    x0 = np.float32(0.8)
    e = rng.standard_normal(n).astype(np.float32)
    z = rng.standard_normal(n).astype(np.float32)
    xt = (np.sqrt(np.float32(a_t)) * x0 + np.sqrt(np.float32(1 - a_t)) * e).astype(np.float32)
    xp = ddim.ddim_step_eta(xt, e, a_t, a_p, eta, z).astype(np.float64)
    assert abs(xp.mean() - math.sqrt(float(a_p)) * 0.8) < 5e-3
    assert abs(xp.var() - (1 - float(a_p))) < 5e-3


def test_stochastic_step_by_hand_and_resumption():
    """With eps = 0 the update is x_prev = sqrt(a_p / a_t) x_t + sigma z (worked by hand in
    float64).  A run resumed at step i from the full run's state, with the same per-step
    draws noise[step], reproduces the full run's tail exactly (draws are indexed by the
    grid step, not by the resumed run's own count)."""
    S = synth.SCHEDULE_SD
    _, a_t, a_p = schedule.step_alphas(30, 50, S)
    xt = np.array([0.5, -1.25, 2.0], np.float32)
    z = np.array([1.0, 0.5, -2.0], np.float32)
    sig = math.sqrt((1 - float(a_p)) / (1 - float(a_t))) * math.sqrt(1 - float(a_t) / float(a_p))
    want = math.sqrt(float(a_p) / float(a_t)) * xt.astype(np.float64) + 0.7 * sig * z
    got = ddim.ddim_step_eta(xt, np.zeros(3, np.float32), a_t, a_p, 0.7, z)
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-7)
    rng = np.random.default_rng(3)
    noise = rng.standard_normal((20, 6)).astype(np.float32)
    x = rng.standard_normal(6).astype(np.float32)
    fn = lambda v, t: ((0.05 * v).astype(np.float32), (0.1 * v + 0.01).astype(np.float32))
    states = {}
    full = ddim.denoise(fn, x, 0, 20, S, 2.0, record=lambda i, v: states.__setitem__(i, v),
                        eta=0.6, noise=noise)
    for i in (3, 11):
        tail = ddim.denoise(fn, states[i], i, 20, S, 2.0, eta=0.6, noise=noise)
        assert np.array_equal(tail, full)
