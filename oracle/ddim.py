"""Classifier-free guidance, the DDIM update and approximate-cache resumption.

Test infrastructure only.  Sec. 4.1: a cache hit at K takes the latent that a
different prompt's run held after its K-th denoising step and runs only the
remaining N - K steps, conditioned on the new prompt.  Sec. 6: the sampler is
DDIM; readings: deterministic (eta = 0), no clipping of the predicted x_0,
guidance eps = eps_u + s (eps_c - eps_u).  All arithmetic is float32.

Sec. 9 suggests changing the denoising seed after a cache hit to keep images
diverse; with a deterministic sampler the seed only enters through x_N, so it
is read as DDIM's stochastic family (Song et al., the update with
sigma = eta sqrt((1 - a_prev)/(1 - a_t)) sqrt(1 - a_t/a_prev) and a fresh
standard normal z per step, which the caller draws from the new seed).
"""
import numpy as np

from . import schedule


def cfg_combine(eps_u, eps_c, s):
    s = np.float32(s)
    return (eps_u + s * (eps_c - eps_u)).astype(np.float32)


def ddim_step(x, eps, a_t, a_prev):
    """One deterministic DDIM update from abar_t to abar_prev (float32)."""
    a_t = np.float32(a_t)
    a_prev = np.float32(a_prev)
    one = np.float32(1.0)
    x0 = (x - np.sqrt(one - a_t) * eps) / np.sqrt(a_t)
    return (np.sqrt(a_prev) * x0 + np.sqrt(one - a_prev) * eps).astype(np.float32)


def ddim_sigma(a_t, a_prev, eta):
    """The noise scale of DDIM's stochastic update from abar_t to abar_prev (float32)."""
    one = np.float32(1.0)
    a_t, a_prev, eta = np.float32(a_t), np.float32(a_prev), np.float32(eta)
    return np.float32(eta * np.sqrt((one - a_prev) / (one - a_t)) * np.sqrt(one - a_t / a_prev))


def ddim_step_eta(x, eps, a_t, a_prev, eta, z):
    """One DDIM update with noise scale sigma(eta) and standard normal draws z (float32)."""
    a_t = np.float32(a_t)
    a_prev = np.float32(a_prev)
    one = np.float32(1.0)
    sigma = ddim_sigma(a_t, a_prev, eta)
    x0 = (x - np.sqrt(one - a_t) * eps) / np.sqrt(a_t)
    dir_ = np.sqrt(max(one - a_prev - sigma * sigma, np.float32(0.0))) * eps
    return (np.sqrt(a_prev) * x0 + dir_ + sigma * z).astype(np.float32)


def denoise(eps_fn, x, K, N, sched, guidance, record=None, eta=0.0, noise=None):
    """Run steps K .. N-1 from latent x (the state after K steps).

    eps_fn(x, t) -> (eps_uncond, eps_cond) for one sample.
    record(i, x) is called with the state after i steps, for i = K .. N.
    noise (optional, [N][*x.shape]): the standard normal draws of each grid step
    for the stochastic update with the given eta.
    Returns x_0 (float32).  K = N returns x unchanged.
    """
    if not (0 <= K <= N):
        raise ValueError("K out of range")
    x = np.asarray(x, dtype=np.float32).copy()
    if record is not None:
        record(K, x.copy())
    for i in range(K, N):
        t, a_t, a_prev = schedule.step_alphas(i, N, sched)
        eu, ec = eps_fn(x, t)
        eps = cfg_combine(eu, ec, guidance)
        if noise is None:
            x = ddim_step(x, eps, a_t, a_prev)
        else:
            x = ddim_step_eta(x, eps, a_t, a_prev, eta, noise[i])
        if record is not None:
            record(i + 1, x.copy())
    return x
