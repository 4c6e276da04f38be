"""GPU parity of the UNet evaluation and the K-skipped DDIM loop (tiny shape).

Bars: per-row epsilon (teacher-forced on the oracle's latent) max-abs <= 1e-2;
final latent relative L2 <= 2e-2 against the float32 oracle.  Resumption from
the state after K steps is the approximate-caching hit path of Sec. 4.1; K = N
returns the cached state unchanged (pure retrieval, Sec. 5.3.1).
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import ddim, schedule
from oracle import unet as U

pytestmark = pytest.mark.gpu

S = synth.SCHEDULE_SD
SCHED = lambda N: (S["T"], N, S["beta_start"], S["beta_end"])
EPS_TOL = 1e-2
X0_TOL = 2e-2


def rel_l2(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.fixture(scope="module")
def tiny():
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("tiny")
    w = synth.make_weights(cfg, 0)
    net = P.NvUNet(cfg, w)
    yield cfg, w, net, U.UNet(cfg, w)
    net.close()


def _ctx(cfg, b, seed):
    return synth.make_contexts(b, cfg["ctx_len"], cfg["ctx_dim"], seed)


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def test_eps_teacher_forced(tiny):
    cfg, _, net, ora = tiny
    B, N = 3, 20
    x = synth.make_latents(B, 4, cfg["H"], cfg["W"], 7)
    cond, unc = _ctx(cfg, B, 11), _ctx(cfg, B, 12)
    steps = [0, 9, 19]
    print("tiny eps parity", flush=True)
    eu, ec = net.nv_unet_eps(t(x), steps, t(cond), t(unc), sched=SCHED(N))
    eu, ec = eu.cpu().numpy(), ec.cpu().numpy()
    for b in range(B):
        ts = schedule.timesteps(N, 1000)[steps[b]]
        ru, rc = ora(x[b], ts, unc[b]), ora(x[b], ts, cond[b])
        du, dc = np.abs(eu[b] - ru).max(), np.abs(ec[b] - rc).max()
        print(f"  b{b} t={ts} maxabs u {du:.2e} c {dc:.2e}", flush=True)
        assert du <= EPS_TOL and dc <= EPS_TOL


def test_eps_teacher_forced_strong_layernorm():
    """Transformer LayerNorms with gains far from 1 and large shifts, and output projections
    scaled up so that the transformer branches weigh on epsilon (in the oracle, dropping the
    shifts or the gains moves epsilon by 0.18 and 0.17 here): the products that fold the
    LayerNorm (gamma-scaled weights, row statistics in the kernel, beta . W in the bias) must
    still match the oracle, which applies the LayerNorm first."""
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("tiny")
    w = dict(synth.make_weights(cfg, 0))
    rng = np.random.default_rng(21)
    for k in list(w):
        if ".ln" in k and k.endswith(".g"):
            w[k] = (2.0 * (1.0 + rng.uniform(-0.5, 0.5, w[k].shape))).astype(np.float32)
        elif ".ln" in k and k.endswith(".b"):
            w[k] = rng.normal(0.0, 1.0, w[k].shape).astype(np.float32)
        elif k.endswith((".attn1.o.w", ".attn2.o.w", ".ff2.w")):
            w[k] = (w[k] * 8.0).astype(np.float32)
    net = P.NvUNet(cfg, w)
    try:
        ora = U.UNet(cfg, w)
        B, N = 2, 20
        x = synth.make_latents(B, 4, cfg["H"], cfg["W"], 17)
        cond, unc = _ctx(cfg, B, 31), _ctx(cfg, B, 32)
        steps = [3, 15]
        print("tiny eps parity, strong LayerNorm parameters", flush=True)
        eu, ec = net.nv_unet_eps(t(x), steps, t(cond), t(unc), sched=SCHED(N))
        eu, ec = eu.cpu().numpy(), ec.cpu().numpy()
        for b in range(B):
            ts = schedule.timesteps(N, 1000)[steps[b]]
            ru, rc = ora(x[b], ts, unc[b]), ora(x[b], ts, cond[b])
            du, dc = np.abs(eu[b] - ru).max(), np.abs(ec[b] - rc).max()
            print(f"  b{b} t={ts} maxabs u {du:.2e} c {dc:.2e}", flush=True)
            assert du <= EPS_TOL and dc <= EPS_TOL
    finally:
        net.close()


def _cached_state(ora, cfg, i, K, N):
    """State after K steps of a full oracle run for cached entry i (own prompt, own x_N)."""
    ctx = _ctx(cfg, 2, 1000 + i)
    xN = synth.make_latents(1, 4, cfg["H"], cfg["W"], 2000 + i)[0]
    states = {}
    ddim.denoise(U.make_eps_fn(ora, ctx[0], ctx[1]), xN, 0, N, S, 7.5,
                 record=lambda j, v: states.__setitem__(j, v))
    return states[K]


@pytest.mark.parametrize("K", [0, 5, 10])
def test_denoise_single(tiny, K):
    cfg, _, net, ora = tiny
    N = 20
    xK = _cached_state(ora, cfg, 3, K, N)
    cond, unc = _ctx(cfg, 1, 21), _ctx(cfg, 1, 22)
    print(f"tiny denoise K={K}", flush=True)
    lat = t(xK[None].copy())
    net.nv_denoise(lat, [K], t(cond), t(unc), guidance=7.5, sched=SCHED(N))
    got = lat.cpu().numpy()[0]
    ref = ddim.denoise(U.make_eps_fn(ora, cond[0], unc[0]), xK, K, N, S, 7.5)
    err = rel_l2(got, ref)
    print(f"  rel-L2 {err:.2e}", flush=True)
    assert err <= X0_TOL


def test_denoise_mixed_k_batch(tiny):
    """One call with per-sample K equals per-sample oracle runs (batch independence)."""
    cfg, _, net, ora = tiny
    N = 20
    Ks = [10, 0, 5, 20, 5]
    xs = np.stack([_cached_state(ora, cfg, i, K, N) for i, K in enumerate(Ks)])
    cond, unc = _ctx(cfg, len(Ks), 31), _ctx(cfg, len(Ks), 32)
    print("tiny mixed-K batch", flush=True)
    lat = t(xs.copy())
    net.nv_denoise(lat, Ks, t(cond), t(unc), guidance=7.5, sched=SCHED(N))
    got = lat.cpu().numpy()
    for b, K in enumerate(Ks):
        ref = ddim.denoise(U.make_eps_fn(ora, cond[b], unc[b]), xs[b], K, N, S, 7.5)
        if K == N:
            np.testing.assert_array_equal(got[b], xs[b])
        else:
            err = rel_l2(got[b], ref)
            print(f"  b{b} K={K} rel-L2 {err:.2e}", flush=True)
            assert err <= X0_TOL


def test_zero_eps_closed_form_on_gpu():
    """conv_out zeroed: eps = 0 and the DDIM loop scales x_K by sqrt(abar_end / abar_tK)."""
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("tiny")
    w = dict(synth.make_weights(cfg, 0))
    w["conv_out.w"] = np.zeros_like(w["conv_out.w"])
    w["conv_out.b"] = np.zeros_like(w["conv_out.b"])
    net = P.NvUNet(cfg, w)
    N, K = 20, 5
    x = synth.make_latents(2, 4, 16, 16, 3)
    cond, unc = _ctx(cfg, 2, 1), _ctx(cfg, 2, 2)
    lat = t(x.copy())
    print("tiny zero-eps closed form", flush=True)
    net.nv_denoise(lat, [K, 0], t(cond), t(unc), sched=SCHED(N))
    ac = schedule.alphas_cumprod64(1000, 0.00085, 0.012)
    ts = schedule.timesteps(N, 1000)
    got = lat.cpu().numpy()
    np.testing.assert_allclose(got[0], x[0] * math.sqrt(ac[0] / ac[ts[K]]), rtol=2e-5)
    np.testing.assert_allclose(got[1], x[1] * math.sqrt(ac[0] / ac[ts[0]]), rtol=2e-5)
    net.close()
