"""Writes sd15_tail_k25.npz with the oracle alone: a cache hit at K = 25 on the
SD-1.5-shaped network, the configuration the benchmark times (Sec. 4.1: the
new prompt resumes from the state another prompt's run held after K steps
and runs the remaining N - K = 25 guided DDIM steps).

  x_k   : the cached prompt's state after 25 of its 50 guided steps, from x_N
          (latent seed 2003, contexts seeds 9 / 10)
  x0    : the oracle's x_0 for the new prompt (contexts seeds 11 / 12) resumed
          from x_k at K = 25
Weights: synth.make_weights(sd15, 0); guidance 7.5; the scaled-linear DDIM
schedule with T = 1000, N = 50.

Usage: python tests/golden/make_sd15_tail.py   (about 30 minutes on 8 cores)
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import synth  # noqa: E402
from oracle import ddim, schedule  # noqa: E402
from oracle import unet as U  # noqa: E402

K, N, GUIDANCE = 25, 50, 7.5
SEEDS = dict(latent=2003, cached_cond=9, cached_uncond=10, cond=11, uncond=12)


def main():
    cfg = synth.unet_config("sd15")
    S = synth.SCHEDULE_SD
    net = U.UNet(cfg, synth.make_weights(cfg, 0))
    ctx = lambda seed: synth.make_contexts(1, 77, 768, seed)[0]
    x = synth.make_latents(1, 4, 64, 64, SEEDS["latent"])[0]
    eps_a = U.make_eps_fn(net, ctx(SEEDS["cached_cond"]), ctx(SEEDS["cached_uncond"]))
    for i in range(K):  # the cached prompt's first K steps
        t, a_t, a_prev = schedule.step_alphas(i, N, S)
        eu, ec = eps_a(x, t)
        x = ddim.ddim_step(x, ddim.cfg_combine(eu, ec, GUIDANCE), a_t, a_prev)
        print(f"cached run step {i + 1}/{K}", flush=True)
    x_k = x.copy()
    eps_b = U.make_eps_fn(net, ctx(SEEDS["cond"]), ctx(SEEDS["uncond"]))
    x0 = ddim.denoise(eps_b, x_k, K, N, S, GUIDANCE,
                      record=lambda i, v: print(f"tail state {i}/{N}", flush=True))
    np.savez_compressed(os.path.join(HERE, "sd15_tail_k25.npz"), x_k=x_k, x0=x0,
                        seeds=np.array([SEEDS[k] for k in sorted(SEEDS)]))
    print("wrote sd15_tail_k25.npz")


if __name__ == "__main__":
    main()
