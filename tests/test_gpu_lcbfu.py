"""GPU parity of the maintained cache (Sec. 5.4): the hole-aware fetch, the
table updates and row compaction that apply the maintainer's plans, and a
whole request stream served through lookup -> hole-aware fetch -> access
counts -> LCBFU eviction / insertion -> generation storing states into the
pool, replayed beside the oracle.

Bars: every K served, every matched row, every plan, the final cache rows,
payload and table are identical to the oracle's; fetched states and moved rows
are bit-exact; states the stream stored agree with a separate full
generation of the same request to relative L2 <= 2e-3 (far below the
difference between neighbouring slots of one trajectory).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import lookup as LK
from oracle.lcbfu import LCBFU

pytestmark = pytest.mark.gpu

SD = synth.SCHEDULE_SD
N = 40
SCHED = (SD["T"], N, SD["beta_start"], SD["beta_end"])
TP = [t for t, _ in synth.THRESHOLDS_PAPER]
KP = [k for _, k in synth.THRESHOLDS_PAPER]
SLOTS = [5, 10, 15, 20, 25]


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _oracle_with_holes(seed, cap=30, ecap=36, steps=80):
    rng = np.random.default_rng(seed)
    o = LCBFU(SLOTS, cap, ecap)
    for _ in range(steps):
        if o.rows and rng.random() < 0.6:
            rows = rng.integers(0, len(o.rows), size=4)
            ks = [o.choose_k(int(r), int(rng.choice(KP + [0, 30]))) for r in rows]
            o.access([int(r) for r in rows], ks)
        else:
            o.insert(int(rng.integers(1, 3)))
    return o


@pytest.mark.parametrize("seed", [0, 1])
def test_gather_pool_hole_choice(seed):
    """K' = the largest stored K' <= K of the matched prompt, the pool state fetched
    bit-exactly; no match, K = 0, or no stored K' <= K -> noise and K' = 0."""
    import paper_2312_04429_amd as P
    o = _oracle_with_holes(seed)
    holes = sum(1 for e in o.rows for s in range(5) if o.state_pool(e, s) < 0)
    print(f"gather_pool seed={seed} rows={len(o.rows)} holes={holes}", flush=True)
    assert holes > 0
    table = np.full((o.ecap, 5), -1, np.int32)
    for e, row in o.table().items():
        table[e] = row
    rng = np.random.default_rng(100 + seed)
    lat = (4, 8, 8)
    pool = rng.standard_normal((o.cap,) + lat).astype(np.float32)
    n = len(o.rows)
    B = 64
    rows = rng.integers(-1, n + 1, size=B)           # -1 and n: no valid match
    ks = rng.choice([0, 3, 5, 7, 10, 12, 15, 20, 22, 25, 40], size=B).astype(np.int32)
    noise = rng.standard_normal((B,) + lat).astype(np.float32)
    payload = np.array(o.rows + [0] * (o.ecap - n), np.int32)
    k_dev = t(ks)
    out = P.nv_gather_pool(t(pool), t(table), SLOTS, t(payload), n, t(rows.astype(np.int64)),
                           k_dev, t(noise))
    got, got_k = out.cpu().numpy(), k_dev.cpu().numpy()
    for b in range(B):
        r = int(rows[b])
        kp = o.choose_k(r, int(ks[b])) if 0 <= r < n else 0
        assert got_k[b] == kp, (b, r, ks[b])
        if kp:
            np.testing.assert_array_equal(got[b], pool[o.state_pool(o.rows[r], SLOTS.index(kp))])
        else:
            np.testing.assert_array_equal(got[b], noise[b])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_plan_application(dtype):
    """Row moves and table records of maintainer plans, applied on the device, give
    the oracle's rows, payload and table bit for bit."""
    import paper_2312_04429_amd as P
    d, cap, ecap = 64, 30, 40
    nat = P.NvLCBFU(SLOTS, cap, ecap)
    o = LCBFU(SLOTS, cap, ecap)
    rng = np.random.default_rng(9)
    emb = rng.standard_normal((400, d)).astype(np.float32)
    bits = synth.to_bf16_bits(emb).view(np.int16) if dtype == "bf16" else emb
    cache = torch.zeros((ecap, d), dtype=torch.int16 if dtype == "bf16" else torch.float32,
                        device="cuda")
    payload = torch.full((ecap,), -1, dtype=torch.int32, device="cuda")
    table = torch.full((ecap, 5), -1, dtype=torch.int32, device="cuda")
    ora_rows = []          # the oracle's vector DB: embedding ids per row
    n, nxt = 0, 0
    moves = 0
    for step in range(60):
        if o.rows and rng.random() < 0.5:
            rows = rng.integers(0, len(o.rows), size=3)
            ks = [o.choose_k(int(r), int(rng.choice(KP))) for r in rows]
            o.access([int(r) for r in rows], ks)
            nat.access(rows, ks)
            continue
        m = int(rng.integers(1, 3))
        p, q = nat.insert(m), o.insert(m)
        assert p["entries"].tolist() == q["entries"]
        for src, dst in q["moves"]:
            ora_rows[dst] = ora_rows[src]
        del ora_rows[q["kept"]:]
        ora_rows += list(range(nxt, nxt + m))
        moves += len(q["moves"])
        P.nv_cache_move_rows(cache, n, payload, t(p["move_src"]), t(p["move_dst"]))
        P.nv_table_update(table, t(p["upd"]))
        n = P.nv_cache_insert(t(emb[nxt:nxt + m]), cache, p["kept"],
                              entry=t(p["entries"]), payload=payload)
        nxt += m
        assert n == len(o.rows)
    print(f"plan application {dtype}: {moves} row moves, {o.dropped} prompts dropped",
          flush=True)
    assert moves > 0
    np.testing.assert_array_equal(cache[:n].cpu().numpy(), bits[ora_rows])
    assert payload[:n].cpu().tolist() == o.rows
    tb = table.cpu().numpy()
    for e in range(ecap):
        want = [o.state_pool(e, s) for s in range(5)]
        assert tb[e].tolist() == want, e


@pytest.fixture(scope="module")
def tiny():
    import paper_2312_04429_amd as P
    cfg = synth.unet_config("tiny")
    net = P.NvUNet(cfg, synth.make_weights(cfg, 0))
    yield cfg, net
    net.close()


def test_maintained_stream(tiny):
    """A request stream through the whole maintained path; the oracle replays the
    lookup, the hole choice and the maintainer on its own copy of the vector DB."""
    import paper_2312_04429_amd as P
    cfg, net = tiny
    d, cap, ecap, B, steps = 64, 40, 48, 4, 30
    lat = (4, cfg["H"], cfg["W"])
    q_all = synth.make_prompt_stream(B * steps, d, 32, p_new=0.1)
    # the empty prompt's encoding, the same for every request
    unc = t(np.repeat(synth.make_contexts(1, cfg["ctx_len"], cfg["ctx_dim"], 5000), B, axis=0))
    conds = synth.make_contexts(B * steps, cfg["ctx_len"], cfg["ctx_dim"], 5001)
    noises = synth.make_latents(B * steps, *lat, 5002)
    nat = P.NvLCBFU(SLOTS, cap, ecap)
    o = LCBFU(SLOTS, cap, ecap)
    cache = torch.zeros((ecap, d), dtype=torch.int16, device="cuda")
    payload = torch.full((ecap,), -1, dtype=torch.int32, device="cuda")
    table = torch.full((ecap, 5), -1, dtype=torch.int32, device="cuda")
    pool = torch.zeros((cap,) + lat, device="cuda")
    ora_cache = np.zeros((0, d), np.uint16)
    owner = {}             # entry -> request that stored it
    n = 0
    served = {0: 0, 5: 0, 10: 0, 15: 0, 20: 0, 25: 0}
    holes_hit = 0
    for step in range(steps):
        rq = list(range(step * B, (step + 1) * B))
        q = q_all[rq]
        print(f"stream step {step} rows={n}", flush=True)
        idx, sim, kk = P.nv_cache_lookup(t(q), cache[:n], TP, KP)
        x = P.nv_gather_pool(pool, table, SLOTS, payload, n, idx, kk, t(noises[rq]))
        idx_h, k_h = idx.cpu().numpy(), kk.cpu().numpy()
        oi, _, ok = LK.lookup(q, ora_cache, TP, KP)
        okp = [o.choose_k(int(i), int(k)) for i, k in zip(oi, ok)]
        assert idx_h.tolist() == oi.tolist() and k_h.tolist() == okp
        holes_hit += sum(1 for a, b in zip(ok, okp) if b < a and b > 0)
        for v in okp:
            served[v] += 1
        nat.access(idx_h, k_h)
        o.access([int(i) for i in oi], okp)
        miss = [b for b in range(B) if k_h[b] == 0]
        dst = np.full((B, 5), -1, np.int32)
        if miss:
            p, pq = nat.insert(len(miss)), o.insert(len(miss))
            assert p["entries"].tolist() == pq["entries"] and p["pools"].tolist() == pq["pools"]
            assert list(zip(p["move_src"].tolist(), p["move_dst"].tolist())) == pq["moves"]
            P.nv_cache_move_rows(cache, n, payload, t(p["move_src"]), t(p["move_dst"]))
            P.nv_table_update(table, t(p["upd"]))
            for i, b in enumerate(miss):
                dst[b] = p["pools"][i]
                owner[int(p["entries"][i])] = rq[b]
            for src, dd in pq["moves"]:
                ora_cache[dd] = ora_cache[src]
            ora_cache = np.concatenate([ora_cache[:pq["kept"]],
                                        synth.to_bf16_bits(q[miss])])
        net.nv_denoise_store_pool(x, k_h.tolist(), t(conds[rq]), unc, pool, SLOTS, dst,
                                  sched=SCHED)
        if miss:
            n = P.nv_cache_insert(t(q[miss]), cache, p["kept"], entry=t(p["entries"]),
                                  payload=payload)
        assert n == len(o.rows) == ora_cache.shape[0]
    print(f"served K: {served}, hole fallbacks {holes_hit}, evicted {o.evicted}, "
          f"dropped {o.dropped}", flush=True)
    assert o.evicted > 0 and o.dropped > 0 and holes_hit > 0
    assert sum(served[k] for k in KP) > 0
    np.testing.assert_array_equal(cache[:n].cpu().numpy().view(np.uint16), ora_cache)
    assert payload[:n].cpu().tolist() == o.rows
    tb = table.cpu().numpy()
    for e in o.rows:
        assert tb[e].tolist() == [o.state_pool(e, s) for s in range(5)]
    # stored states: a separate full generation of the storing request
    pl = pool.cpu().numpy()
    live = [(e, s) for e in o.rows for s in range(5) if o.state_pool(e, s) >= 0]
    for e, s in live[:: max(1, len(live) // 6)]:
        r = owner[e]
        store = torch.zeros((1, 5) + lat, device="cuda")
        xr = t(noises[r:r + 1])
        net.nv_denoise_store(xr, [0], t(conds[r:r + 1]), unc[:1], store, SLOTS, [0],
                             sched=SCHED)
        ref = store[0, s].cpu().numpy()
        err = float(np.linalg.norm(pl[o.state_pool(e, s)] - ref) / np.linalg.norm(ref))
        print(f"  entry {e} (request {r}) K={SLOTS[s]} rel-L2 {err:.2e}", flush=True)
        assert err <= 2e-3
