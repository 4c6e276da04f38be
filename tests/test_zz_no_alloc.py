"""nv_cache_lookup_static (the lookup on the library's own scratch array, for
callers that cannot allocate) against nv_cache_lookup on a caller workspace:
bit-identical indices, similarity bits and K on consecutive calls that share
the array, a large bf16 cache first and then a smaller f32 one (whose result
is also checked against the oracle), and the large one again."""
import numpy as np
import pytest
import torch

import synth
from oracle import lookup as LK

pytestmark = pytest.mark.gpu

THR = [t for t, _ in synth.THRESHOLDS_PAPER]
KV = [k for _, k in synth.THRESHOLDS_PAPER]


def _same(a, b):
    ia, sa, ka = (x.cpu() for x in a)
    ib, sb, kb = (x.cpu() for x in b)
    assert torch.equal(ia, ib)
    assert torch.equal(sa.view(torch.int32), sb.view(torch.int32))
    assert torch.equal(ka, kb)


def test_static_lookup_matches_workspace_lookup_on_consecutive_calls():
    import paper_2312_04429_amd as P
    from paper_2312_04429_amd import _native as N
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    big = synth.make_cache(200_000, 768, 1000, 0.05, 51, "bf16")
    qa = np.concatenate([synth.make_queries_at_sims(synth.cache_rows_f32(big, [7 + 4001 * i]),
                                                    [0.96 - 0.01 * i], 60 + i)
                         for i in range(20)] +
                        [synth.make_cluster_queries(20, 768, 1000, 0.05, 51, 61)])
    assert qa.shape == (40, 768)
    need_a = N.lib.nv_cache_lookup_workspace(40, 200_000, 768)
    assert 0 < need_a <= N.NV_LOOKUP_STATIC_BYTES
    small = synth.make_cache(1500, 64, 16, 0.1, 52, "f32")
    qb = synth.make_queries_at_sims(small[[3, 900, 1499]], [0.97, 0.88, 0.7], 62)
    ca, qa_d, cb, qb_d = t(big), t(qa), t(small), t(qb)
    print("static lookup: 40 queries x 200000 x 768 bf16", flush=True)
    ra = P.nv_cache_lookup_static(qa_d, ca, THR, KV)
    _same(ra, P.nv_cache_lookup(qa_d, ca, THR, KV))
    print("static lookup: 3 queries x 1500 x 64 f32 (smaller, same array)", flush=True)
    rb = P.nv_cache_lookup_static(qb_d, cb, THR, KV)
    _same(rb, P.nv_cache_lookup(qb_d, cb, THR, KV))
    oi, osim, ok = LK.lookup(qb, small, THR, KV)
    assert rb[0].cpu().numpy().tolist() == list(oi)
    assert rb[1].cpu().numpy().view(np.int32).tolist() == np.asarray(osim, np.float32).view(
        np.int32).tolist()
    assert rb[2].cpu().numpy().tolist() == list(ok)
    print("static lookup: the large call again after the small one", flush=True)
    _same(P.nv_cache_lookup_static(qa_d, ca, THR, KV), ra)
