"""Denoise steps replayed from captured HIP graphs against the same steps
launched kernel by kernel (nv_unet_set_options without NV_UNET_GRAPHS):
bit-identical x_0.

The replays run several times per handle with other GPU work and
synchronisations between them, across calls that change the active row count
(a mixed-K batch leaves samples behind as they finish, so each row count has
its own graph), the guidance, eta with its noise, the batch size, and the
snapshot copies of the miss path between replays; on the tiny network and on
the SD-1.5-shaped network of the benchmark."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

S = synth.SCHEDULE_SD


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _run(net, x, ks, cond, unc, sched, graphs, guidance=7.5, eta=None, noise=None):
    net.set_options(graphs=graphs)
    lat = t(x.copy())
    if eta is None:
        net.nv_denoise(lat, ks, t(cond), t(unc), guidance=guidance, sched=sched)
    else:
        net.nv_denoise_eta(lat, ks, t(cond), t(unc), eta, noise, guidance=guidance, sched=sched)
    return lat.cpu().numpy()


def _other_work():
    a = torch.randn(1 << 20, device="cuda")
    (a * 2.0 + 1.0).sum().item()
    torch.cuda.synchronize()


def test_graph_replay_matches_eager_tiny():
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("tiny")
    net = P.NvUNet(cfg, synth.make_weights(cfg, 0))
    N = 20
    sched = (S["T"], N, S["beta_start"], S["beta_end"])
    ks = [10, 0, 5, 20, 5]
    x = synth.make_latents(5, 4, cfg["H"], cfg["W"], 31)
    cond = synth.make_contexts(5, cfg["ctx_len"], cfg["ctx_dim"], 32)
    unc = synth.make_contexts(5, cfg["ctx_len"], cfg["ctx_dim"], 33)
    ref = _run(net, x, ks, cond, unc, sched, False)
    for rep in range(3):
        got = _run(net, x, ks, cond, unc, sched, True)
        np.testing.assert_array_equal(got, ref, err_msg=f"replay {rep}")
        _other_work()
    # a new guidance rebuilds the graphs
    ref2 = _run(net, x, ks, cond, unc, sched, False, guidance=3.0)
    assert np.abs(ref2 - ref).max() > 1e-3
    np.testing.assert_array_equal(_run(net, x, ks, cond, unc, sched, True, guidance=3.0), ref2)
    # a smaller batch (another plan and workspace) and back
    ref3 = _run(net, x[:2], ks[:2], cond[:2], unc[:2], sched, False)
    np.testing.assert_array_equal(_run(net, x[:2], ks[:2], cond[:2], unc[:2], sched, True), ref3)
    np.testing.assert_array_equal(_run(net, x, ks, cond, unc, sched, True), ref)
    # stochastic update: eta and the noise pointer enter the captured step
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    noise = torch.randn((5, N, 4, cfg["H"], cfg["W"]), generator=g, device="cuda")
    ref4 = _run(net, x, ks, cond, unc, sched, False, eta=0.5, noise=noise)
    for rep in range(2):
        np.testing.assert_array_equal(_run(net, x, ks, cond, unc, sched, True, eta=0.5,
                                           noise=noise), ref4)
        _other_work()
    # snapshots between replays (miss path)
    store_e = torch.zeros((5, 2, 4, cfg["H"], cfg["W"]), device="cuda")
    store_g = torch.zeros_like(store_e)
    for graphs, store in ((False, store_e), (True, store_g)):
        net.set_options(graphs=graphs)
        lat = t(x.copy())
        net.nv_denoise_store(lat, ks, t(cond), t(unc), store, [5, 10], [0, 1, 2, 3, 4],
                             sched=sched)
        if graphs:
            np.testing.assert_array_equal(lat.cpu().numpy(), ref)
    assert torch.equal(store_e, store_g)
    net.close()


def test_graph_replay_matches_eager_sd15():
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("sd15")
    print("generating SD-1.5-shaped weights", flush=True)
    net = P.NvUNet(cfg, synth.make_weights(cfg, 0))
    sched = (S["T"], 50, S["beta_start"], S["beta_end"])
    x = synth.make_latents(2, 4, 64, 64, 41)
    cond = synth.make_contexts(2, 77, 768, 42)
    unc = synth.make_contexts(2, 77, 768, 43)
    print("sd15 batch 1, K = 46 eager", flush=True)
    ref = _run(net, x[:1], [46], cond[:1], unc[:1], sched, False)
    for rep in range(2):
        print(f"sd15 batch 1 graph replay {rep}", flush=True)
        np.testing.assert_array_equal(_run(net, x[:1], [46], cond[:1], unc[:1], sched, True), ref)
        _other_work()
    print("sd15 batch 2 mixed K eager / graphs", flush=True)
    ref2 = _run(net, x, [47, 45], cond, unc, sched, False)
    np.testing.assert_array_equal(_run(net, x, [47, 45], cond, unc, sched, True), ref2)
    assert np.isfinite(ref2).all()
    net.close()

