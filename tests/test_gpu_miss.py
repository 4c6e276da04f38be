"""GPU parity of the cache-miss side of Alg. 1 (Sec. 4.3): a request without a
suitable cache runs the full generation, its states after each K of the
selector table are stored for later hits, and its embedding joins the cache.

Bars: stored states against the oracle's states after the same number of
steps (relative L2 <= 2e-2, the final-latent bar); the state a sample was
given and the cache rows written are bit-exact; a lookup of the inserted
prompt hits its own row at the top K, and resuming from the stored state
reproduces the full run's x_0 bit for bit (same kernels on the same inputs).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import ddim
from oracle import lookup as LK
from oracle import unet as U

pytestmark = pytest.mark.gpu

S = synth.SCHEDULE_SD
N = 20
SCHED = (S["T"], N, S["beta_start"], S["beta_end"])
TT = [t for t, _ in synth.THRESHOLDS_TINY]
KT = [k for _, k in synth.THRESHOLDS_TINY]
SLOTS = [5, 10]


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def rel_l2(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.fixture(scope="module")
def tiny():
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("tiny")
    w = synth.make_weights(cfg, 0)
    net = P.NvUNet(cfg, w)
    yield cfg, net, U.UNet(cfg, w)
    net.close()


def test_denoise_store_states_match_oracle(tiny):
    cfg, net, ora = tiny
    x = synth.make_latents(2, 4, cfg["H"], cfg["W"], 4000)
    cond = synth.make_contexts(2, cfg["ctx_len"], cfg["ctx_dim"], 4001)
    unc = synth.make_contexts(2, cfg["ctx_len"], cfg["ctx_dim"], 4002)
    k = [0, 5]
    store = torch.zeros(4, len(SLOTS), 4, cfg["H"], cfg["W"], device="cuda")
    print("tiny denoise with stored states", flush=True)
    lat = t(x.copy())
    net.nv_denoise_store(lat, k, t(cond), t(unc), store, SLOTS, [3, 1], sched=SCHED)
    ref_lat = t(x.copy())
    net.nv_denoise(ref_lat, k, t(cond), t(unc), sched=SCHED)
    assert torch.equal(lat, ref_lat)  # storing does not change the generation
    st = store.cpu().numpy()
    for b, e in ((0, 3), (1, 1)):
        states = {}
        ddim.denoise(U.make_eps_fn(ora, cond[b], unc[b]), x[b], k[b], N, S, 7.5,
                     record=lambda i, v: states.__setitem__(i, v))
        for q, ks in enumerate(SLOTS):
            if ks == k[b]:
                np.testing.assert_array_equal(st[e, q], x[b])  # the state it was given
            else:
                err = rel_l2(st[e, q], states[ks])
                print(f"  sample {b} slot K={ks} rel-L2 {err:.2e}", flush=True)
                assert err <= 2e-2
    assert not st[0].any() and not st[2].any()  # entries nobody wrote


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_cache_insert(dtype):
    import paper_2312_04429_amd as P
    print(f"cache insert {dtype}", flush=True)
    rng = np.random.default_rng(5)
    rows = rng.standard_normal((3, 64)).astype(np.float32)
    cap, n = 10, 4
    if dtype == "bf16":
        cache = torch.zeros(cap, 64, dtype=torch.int16, device="cuda")
    else:
        cache = torch.zeros(cap, 64, dtype=torch.float32, device="cuda")
    payload = torch.full((cap,), -7, dtype=torch.int32, device="cuda")
    entry = torch.tensor([11, 12, 13], dtype=torch.int32, device="cuda")
    n2 = P.nv_cache_insert(t(rows), cache, n, entry=entry, payload=payload)
    assert n2 == 7
    got = cache.cpu().numpy()
    want = synth.to_bf16_bits(rows).view(np.int16) if dtype == "bf16" else rows
    np.testing.assert_array_equal(got[4:7], want)
    assert not got[:4].any() and not got[7:].any()
    assert payload.cpu().tolist() == [-7] * 4 + [11, 12, 13] + [-7] * 3
    with pytest.raises(Exception):
        P.nv_cache_insert(t(rows), cache, 8)  # past the capacity


def test_miss_insert_hit_closed_loop(tiny):
    """Miss -> full generation storing its states -> insert -> the same prompt now
    hits its own row at the top K, and resuming from the stored state gives the
    full run's x_0 exactly."""
    import paper_2312_04429_amd as P
    cfg, net, _ = tiny
    w = synth.WORKLOADS["tiny"]
    cache_np = synth.make_cache(w["n_cache"], w["d"], w["clusters"], w["sigma"], w["cache_seed"],
                                "f32")
    cap = w["n_cache"] + 4
    cache = torch.zeros(cap, w["d"], dtype=torch.float32, device="cuda")
    cache[: w["n_cache"]] = t(cache_np)
    payload = torch.zeros(cap, dtype=torch.int32, device="cuda")
    rng = np.random.default_rng(77)
    q = rng.standard_normal((1, w["d"])).astype(np.float32)
    q /= np.linalg.norm(q)
    n = w["n_cache"]
    print("closed loop: lookup (miss)", flush=True)
    idx, sim, kk = P.nv_cache_lookup(t(q), cache[:n], TT, KT)
    oi, os_, ok = LK.lookup(q, cache_np, TT, KT)
    assert idx.item() == oi[0] and kk.item() == ok[0] == 0  # a miss
    x = synth.make_latents(1, 4, cfg["H"], cfg["W"], 4100)
    cond = synth.make_contexts(1, cfg["ctx_len"], cfg["ctx_dim"], 4101)
    unc = synth.make_contexts(1, cfg["ctx_len"], cfg["ctx_dim"], 4102)
    store = torch.zeros(2, len(SLOTS), 4, cfg["H"], cfg["W"], device="cuda")
    full = t(x.copy())
    net.nv_denoise_store(full, [0], t(cond), t(unc), store, SLOTS, [1], sched=SCHED)
    n = P.nv_cache_insert(t(q), cache, n, entry=torch.tensor([1], dtype=torch.int32,
                                                              device="cuda"), payload=payload)
    print("closed loop: lookup (hit)", flush=True)
    idx, sim, kk = P.nv_cache_lookup(t(q), cache[:n], TT, KT)
    assert idx.item() == n - 1 and kk.item() == max(KT)
    resumed = P.nv_gather_states(store, SLOTS, payload[:n], n, idx, kk, t(x))
    net.nv_denoise(resumed, kk.cpu().tolist(), t(cond), t(unc), sched=SCHED)
    assert torch.equal(resumed, full)
