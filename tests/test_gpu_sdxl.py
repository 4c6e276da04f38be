"""GPU parity at the SDXL topology (Sec. 2.1 latent-diffusion UNet in the SDXL
configuration: three levels, transformer depth 0 / 2 / 10 and a depth-10
middle block, head_dim 64, 77 x 2048 context and a 1280-d pooled vector added
to the time embedding).

Bars as for the other shapes: per-row epsilon max-abs <= 1e-2 (teacher-forced
on the oracle's latent) and final-latent relative L2 <= 2e-2 after a short
K-skipped run, both against the float32 oracle with the same weights.  The
narrow variant keeps the full topology with 64 / 128 / 256 channels (and a
256-d pooled vector, the width of its time embedding) on a 32 x 32 latent so
the oracle runs in seconds; the full-size check compares one
guided row of the 128 x 128, 2.56B-parameter network.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import ddim, schedule
from oracle import unet as U

pytestmark = pytest.mark.gpu

S = synth.SCHEDULE_SD
SCHED = (S["T"], 50, S["beta_start"], S["beta_end"])
NARROW = dict(ch=(64, 128, 256), H=32, W=32, pooled_dim=256)  # pooled vector = 4 ch[0] wide


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.fixture(scope="module")
def narrow():
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("sdxl", **NARROW)
    w = synth.make_weights(cfg, 1)
    net = P.NvUNet(cfg, w)
    yield cfg, net, U.UNet(cfg, w)
    net.close()


def _inputs(cfg, b, seed):
    x = synth.make_latents(b, 4, cfg["H"], cfg["W"], seed)
    cond = synth.make_contexts(b, 77, 2048, seed + 1)
    unc = synth.make_contexts(b, 77, 2048, seed + 2)
    pooled = synth.make_pooled(b, cfg["pooled_dim"], seed + 3)
    return x, cond, unc, pooled


def test_eps_teacher_forced_sdxl_narrow(narrow):
    cfg, net, ora = narrow
    x, cond, unc, pooled = _inputs(cfg, 2, 3000)
    steps = [0, 37]
    print("sdxl-narrow eps", flush=True)
    eu, ec = net.nv_unet_eps(t(x), steps, t(cond), t(unc), pooled=t(pooled), sched=SCHED)
    eu, ec = eu.cpu().numpy(), ec.cpu().numpy()
    for b in range(2):
        ts = schedule.timesteps(50, 1000)[steps[b]]
        ru = ora(x[b], ts, unc[b], pooled=pooled[b])
        rc = ora(x[b], ts, cond[b], pooled=pooled[b])
        du, dc = float(np.abs(eu[b] - ru).max()), float(np.abs(ec[b] - rc).max())
        print(f"  b{b} t={ts} max-abs u {du:.3e} c {dc:.3e}", flush=True)
        assert du <= 1e-2 and dc <= 1e-2


def test_pooled_vector_reaches_the_output(narrow):
    """Changing only the pooled vector changes epsilon on both sides alike."""
    cfg, net, ora = narrow
    x, cond, unc, pooled = _inputs(cfg, 1, 3100)
    p2 = pooled * -1.0
    e1, _ = net.nv_unet_eps(t(x), [10], t(cond), t(unc), pooled=t(pooled), sched=SCHED)
    e2, _ = net.nv_unet_eps(t(x), [10], t(cond), t(unc), pooled=t(p2), sched=SCHED)
    d_gpu = (e1 - e2).cpu().numpy()[0]
    ts = schedule.timesteps(50, 1000)[10]
    d_ora = ora(x[0], ts, unc[0], pooled=pooled[0]) - ora(x[0], ts, unc[0], pooled=p2[0])
    print(f"sdxl-narrow pooled sensitivity |d| {np.abs(d_ora).max():.3e}", flush=True)
    assert np.abs(d_ora).max() > 1e-3
    assert np.abs(d_gpu - d_ora).max() <= 2e-2


def test_denoise_tail_sdxl_narrow(narrow):
    """Four guided steps from a cached state at K = 46, batch of two with
    different pooled vectors, against the oracle."""
    cfg, net, ora = narrow
    K = 46
    xK, cond, unc, pooled = _inputs(cfg, 2, 3200)
    lat = t(xK.copy())
    print("sdxl-narrow denoise K=46", flush=True)
    net.nv_denoise(lat, [K, K], t(cond), t(unc), pooled=t(pooled), guidance=7.5, sched=SCHED)
    got = lat.cpu().numpy()
    for b in range(2):
        ref = ddim.denoise(U.make_eps_fn(ora, cond[b], unc[b], pooled=pooled[b]), xK[b], K, 50,
                           S, 7.5)
        err = float(np.linalg.norm(got[b] - ref) / np.linalg.norm(ref))
        print(f"  b{b} rel-L2 {err:.3e}", flush=True)
        assert err <= 2e-2


def test_eps_full_size_sdxl_one_row():
    """Full SDXL shape (4 x 128 x 128 latent, 2.56B parameters): the conditional
    epsilon of one guided evaluation against the oracle."""
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("sdxl")
    print("generating SDXL-shaped weights", flush=True)
    w = synth.make_weights(cfg, 0)
    net = P.NvUNet(cfg, w)
    try:
        x, cond, unc, pooled = _inputs(cfg, 1, 3300)
        print("sdxl full-size eps (GPU)", flush=True)
        _, ec = net.nv_unet_eps(t(x), [20], t(cond), t(unc), pooled=t(pooled), sched=SCHED)
        ec = ec.cpu().numpy()[0]
    finally:
        net.close()
    ts = schedule.timesteps(50, 1000)[20]
    print("sdxl full-size eps (oracle, one row)", flush=True)
    rc = U.UNet(cfg, w)(x[0], ts, cond[0], pooled=pooled[0])
    dc = float(np.abs(ec - rc).max())
    print(f"  max-abs c {dc:.3e}", flush=True)
    assert dc <= 1e-2
