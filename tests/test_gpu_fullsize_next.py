"""Full-size checks of the maintained cache and the IVF index, at the sizes the
benchmark runs them (properties that hold at any size, and sampled canonical
rescoring by the oracle):

* LCBFU at the paper's operating point (300k prompts, 1.5M states of SD-1.5
  latents, 98 GB pool): over a request stream, every served K' is a stored slot
  at or below the selector's K, the fetched latent is the pool state the host
  maintainer's table names, the device table and payload stay equal to the
  maintainer's, and moved rows carry their original embeddings;
* IVF over 10M x 768 (4096 lists, one Lloyd step): every returned row lies in a
  probed list, its similarity is the oracle's canonical score of that row, its K
  follows the selector, and no sampled row of the probed lists beats it.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import lookup as LK

pytestmark = pytest.mark.gpu

TP = [t for t, _ in synth.THRESHOLDS_PAPER]
KP = [k for _, k in synth.THRESHOLDS_PAPER]
SLOTS = sorted(KP)
BAND = {25: 0.97, 20: 0.925, 15: 0.875, 10: 0.80, 5: 0.70}


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _bits(rows):
    return rows.view(torch.int16).cpu().numpy().view(np.uint16)


def test_lcbfu_stream_at_full_size():
    import paper_2312_04429_amd as P
    wl = synth.WORKLOADS["sd15_lcbfu"]
    n0, cap, d = wl["n_prompts"], wl["state_capacity"], wl["d"]
    lat = (4, 64, 64)
    dev = torch.device("cuda")
    print(f"lcbfu full size: {n0} prompts, {cap} states", flush=True)
    cache = torch.empty((cap, d), dtype=torch.bfloat16, device=dev)
    cache[:n0] = synth.make_cache_device(n0, d, wl["clusters"], wl["sigma"], wl["cache_seed"], dev)
    pool = torch.empty((cap,) + lat, dtype=torch.float32, device=dev)
    for i in range(0, cap, 1 << 16):
        pool[i:i + (1 << 16)].normal_()
    table = torch.full((cap, 5), -1, dtype=torch.int32, device=dev)
    payload = torch.full((cap,), -1, dtype=torch.int32, device=dev)
    lc = P.NvLCBFU(SLOTS, cap, cap)
    for i in range(0, n0, 100_000):
        plan = lc.insert(100_000)
        P.nv_table_update(table, t(plan["upd"]))
        payload[i:i + 100_000] = t(plan["entries"])
    rng = np.random.default_rng(wl["access_seed"])
    lc.access(np.minimum((n0 * rng.random(wl["prefill_accesses"]) ** 3).astype(np.int64), n0 - 1),
              rng.choice(SLOTS, size=wl["prefill_accesses"]).astype(np.int32))
    # a stream with many misses and rewordings of recently inserted prompts
    steps = 60
    rq = np.random.default_rng(7)
    n = n0
    noise = torch.randn((1,) + lat, device=dev)
    lws_bytes = P.nv_cache_lookup_workspace(1, cap, d)
    own, addr = P.workspace(lws_bytes, dev)
    inserted = []          # (row at insertion time, float32 embedding)
    moves = served_hits = 0
    for step in range(steps):
        if inserted and rq.random() < 0.5:
            q = synth.make_queries_at_sims(inserted[rq.integers(0, len(inserted))][1][None],
                                           [BAND[int(rq.choice(SLOTS))]], step)
        elif rq.random() < 0.5:
            r = int(rq.integers(0, n))
            q = synth.make_queries_at_sims(synth.from_bf16_bits(_bits(cache[r:r + 1])),
                                           [BAND[int(rq.choice(SLOTS))]], step)
        else:
            q = synth.make_prompt_stream(1, d, 1000 + step, p_new=1.0)
        dq = t(q.astype(np.float32))
        idx, sim, kk = P.nv_cache_lookup(dq, cache[:n], TP, KP, ws=(own, addr, lws_bytes))
        k_sel = int(kk.item())
        x = P.nv_gather_pool(pool, table, SLOTS, payload, n, idx, kk, noise)
        i_h, k_h = int(idx.item()), int(kk.item())
        assert k_h == 0 or (k_h in SLOTS and k_h <= k_sel)
        ht, hrows, _ = lc.export()
        if k_h:
            e = int(hrows[i_h])
            want = ht[e][SLOTS.index(k_h)]
            # the largest stored slot at or below the selector's K
            stored = [SLOTS[s] for s in range(5) if ht[e][s] >= 0 and SLOTS[s] <= k_sel]
            assert k_h == max(stored)
            assert torch.equal(x[0], pool[int(want)])
            served_hits += 1
        else:
            assert torch.equal(x, noise)
        lc.access([i_h], [k_h])
        if k_h == 0:
            plan = lc.insert(1)
            if len(plan["move_src"]):
                src_rows = cache[t(plan["move_src"])].clone()
                P.nv_cache_move_rows(cache, n, payload, t(plan["move_src"]), t(plan["move_dst"]))
                assert torch.equal(cache[t(plan["move_dst"])], src_rows)
                moves += len(plan["move_src"])
            P.nv_table_update(table, t(plan["upd"]))
            n = P.nv_cache_insert(dq, cache, plan["kept"], entry=t(plan["entries"]),
                                  payload=payload)
            inserted.append((n - 1, q[0]))
            touched = plan["upd"][:, 0]
            ht, hrows, _ = lc.export()
            assert np.array_equal(table[t(touched.astype(np.int64))].cpu().numpy(), ht[touched])
    ht, hrows, _ = lc.export()
    assert np.array_equal(payload[:n].cpu().numpy(), hrows)
    print(f"  {steps} requests: {served_hits} served from the pool, {moves} row moves, "
          f"info {lc.info()}", flush=True)
    assert served_hits > 0 and lc.info()["evicted"] > 0


def test_ivf_at_10m_rows():
    import paper_2312_04429_amd as P
    wl = synth.WORKLOADS["retrieval_heavy"]
    n, d = wl["n_cache"], wl["d"]
    dev = torch.device("cuda")
    print(f"ivf full size: {n} x {d}", flush=True)
    cache = synth.make_cache_device(n, d, wl["clusters"], wl["sigma"], wl["cache_seed"], dev)
    init = np.random.default_rng(wl["cache_seed"] + 7).choice(n, 4096, replace=False)
    index = P.NvIVF(cache, init, 1)
    rng = np.random.default_rng(3)
    planted = rng.integers(0, n, 16)
    rows = synth.from_bf16_bits(_bits(cache[t(planted)]))
    q = np.concatenate([synth.make_queries_at_sims(rows, rng.uniform(0.9, 0.999, 16), 4),
                        synth.make_prompt_stream(16, d, 5, p_new=1.0)]).astype(np.float32)
    gi, gs, gk, gp = index.search(t(q), 32, TP, KP, probed=True)
    gi, gs, gk, gp = (v.cpu().numpy() for v in (gi, gs, gk, gp))
    lists = index.lists
    off = index.offsets.cpu().numpy()
    for j in range(len(q)):
        assert gi[j] >= 0
        assert int(lists[int(gi[j])].item()) in set(gp[j].tolist())
        s = LK.canonical_score_rows(q[j], _bits(cache[int(gi[j]):int(gi[j]) + 1]), [0])[0]
        assert gs[j] == np.float32(s) and gk[j] == LK.select_k(np.float32(s), TP, KP)
        # 4000 rows sampled from the probed lists: none beats the answer
        pos = np.concatenate([np.arange(off[l], off[l + 1]) for l in gp[j]])
        samp = rng.choice(pos, min(4000, len(pos)), replace=False)
        ids = index.perm[t(samp.astype(np.int64))].cpu().numpy()
        sc = LK.canonical_scores(q[j], _bits(index.rows[t(samp.astype(np.int64))]))
        assert np.all((sc < s) | ((sc == s) & (ids >= gi[j])))
    print(f"  32 queries checked; K of the planted half: {gk[:16].tolist()}", flush=True)
