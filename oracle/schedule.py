"""DDIM timestep grid and cumulative alpha table (test infrastructure only).

Sec. 2.1 gives the forward process q(x_t | x_{t-1}) = N(sqrt(1 - beta_t) x_{t-1},
beta_t I) over T steps and the sampler that visits N of them, one every T/N
steps; Sec. 6 names DDIM with N = 50.  Readings (the paper does not print the
schedule): latent-diffusion "scaled linear" betas, T = 1000,
  beta_t = (sqrt(b0) + (sqrt(b1) - sqrt(b0)) * t / (T - 1))^2,  t = 0 .. T-1,
  abar_t = prod_{s <= t} (1 - beta_s)   (float64, then rounded to float32),
  grid t_i = (N - 1 - i) * (T / N) + 1, i = 0 .. N-1 (981, 961, ..., 1 for N = 50),
and step i moves t_i -> t_{i+1}; after the last grid point the target is
abar_0 (not 1).
"""
import numpy as np


def betas(T, beta_start, beta_end):
    t = np.arange(T, dtype=np.float64)
    r0, r1 = np.sqrt(beta_start), np.sqrt(beta_end)
    return (r0 + (r1 - r0) * t / (T - 1)) ** 2


def alphas_cumprod64(T, beta_start, beta_end):
    a = 1.0 - betas(T, beta_start, beta_end)
    out = np.empty(T, dtype=np.float64)
    acc = 1.0
    for i in range(T):
        acc *= a[i]
        out[i] = acc
    return out


def alphas_cumprod(T, beta_start, beta_end):
    return alphas_cumprod64(T, beta_start, beta_end).astype(np.float32)


def timesteps(N, T):
    if T % N != 0:
        raise ValueError("T must be a multiple of N")
    stride = T // N
    return [(N - 1 - i) * stride + 1 for i in range(N)]


def step_alphas(i, N, sched):
    """(t_i, abar_t, abar_prev) as float32 for step index i of an N-step run."""
    T = sched["T"]
    ac = alphas_cumprod(T, sched["beta_start"], sched["beta_end"])
    ts = timesteps(N, T)
    t = ts[i]
    prev = t - T // N
    a_prev = ac[prev] if prev >= 0 else ac[0]
    return t, ac[t], a_prev
