"""GPU parity of the attention kernel (the UNet's self- and cross-attention,
Sec. 2.1) against the oracle's float32 attention on the same float16-valued
inputs, at the head dims of the configurations (16 tiny, 40 / 80 / 160
SD-1.5, 64 SDXL), the 77-token context with its padded V^T rows, ragged
query / key counts, and each launch form (one query block per wave, with two
key sets splitting every key block for 80-dim heads over at most 256
workgroups of 64 queries and for 160-dim heads on small grids; two query
blocks per wave, with eight query waves sharing each key block for 40-dim
heads: two key sets of eight waves at up to 512 four-wave workgroups over more
than 128 keys, as at batch 1 over 4,096 queries, 128-key blocks at that grid
size otherwise, 64-key blocks beyond; two with four waves for the other head
dims).  The key-set cases include slices that hold a single key or none.

The peaked-score cases drive the online softmax through its rescale branch:
the kernel keeps a per-query reference maximum and moves it (multiplying the
running sum and the output accumulators by 2^(old - new)) only when a later
key block scores more than 2^8 above it.  Standard-normal inputs never get
there after the first block, so these cases plant keys aligned with chosen
queries in later key blocks (and, in the "hot" kind, scale every query), for
every launch form of every head dim."""
import numpy as np
import pytest
import torch

from oracle import unet as U

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rows,S,L,heads,dh", [(2, 300, 77, 8, 40), (2, 256, 256, 8, 40),
                                               (1, 200, 130, 8, 80), (2, 64, 77, 8, 160),
                                               (1, 128, 256, 4, 80), (2, 70, 200, 2, 16),
                                               (2, 130, 8, 4, 16), (1, 128, 77, 10, 64),
                                               (1, 96, 100, 2, 32), (1, 64, 64, 2, 128),
                                               (1, 200, 333, 8, 40), (1, 512, 1000, 8, 40),
                                               (2, 2048, 333, 8, 40), (3, 4096, 200, 8, 40),
                                               (16, 256, 256, 8, 160), (16, 256, 77, 8, 160),
                                               (16, 1024, 77, 8, 80), (2, 4096, 4096, 8, 40),
                                               (1, 2000, 1000, 16, 40), (2, 2048, 128, 8, 40),
                                               (1, 128, 20, 4, 80), (2, 1000, 999, 8, 80),
                                               (1, 100, 33, 2, 160), (1, 64, 20, 2, 160),
                                               (2, 256, 256, 8, 160), (1, 4096, 130, 8, 40),
                                               (2, 1024, 1024, 8, 80)])
def test_attention(rows, S, L, heads, dh):
    print(f"op attention rows={rows} S={S} L={L} heads={heads} dh={dh}", flush=True)
    C = heads * dh
    rng = np.random.default_rng(S + L + dh)
    h = lambda a: a.astype(np.float16)
    q = h(rng.standard_normal((rows, S, C)))
    k = h(rng.standard_normal((rows, L, C)))
    v = h(rng.standard_normal((rows, L, C)))
    _check(q, k, v, heads, 1.0 / np.sqrt(dh), 4e-3)


def _check(q, k, v, heads, scale, atol):
    import paper_2312_04429_amd as P
    rows, S, C = q.shape
    L = k.shape[1]
    dh = C // heads
    Lp = (L + 7) // 8 * 8
    vt = np.zeros((C, rows * Lp), dtype=np.float16)
    for r in range(rows):
        vt[:, r * Lp:r * Lp + L] = v[r].T
    vt[:, :] = np.where(np.arange(rows * Lp)[None, :] % Lp >= L, np.float16(np.nan), vt)  # unused keys
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    got = P.nv_op_attention(t(q), t(k), t(vt), heads, scale, L=L, vt_row=Lp)
    got = got.float().cpu().numpy()
    # the oracle's attention scales by 1/sqrt(dh); other scales enter through q
    qs = np.float32(scale * np.sqrt(dh))
    for r in range(rows):
        ref = U.attention(q[r].astype(np.float32) * qs, k[r].astype(np.float32),
                          v[r].astype(np.float32), heads)
        np.testing.assert_allclose(got[r], ref, rtol=0, atol=atol)


# Launch forms (the launcher's rule over wgs2 = ceil(S / 128) * heads * rows):
# wgs2 < 256 -> one query block per wave: 80-dim heads with at most 256
# workgroups of 64 queries in two key sets of four waves on 64-key slices,
# 160-dim heads in workgroups of 32 queries with two key sets of two waves on
# 32-key slices, otherwise four waves with 64-key blocks; wgs2 >= 256 -> two
# query blocks per wave: 40-dim heads with eight query waves (256 queries),
# up to wgs2 = 512 in two key sets on 64-key slices when L > 128 (128-key
# blocks otherwise) and with 64-key blocks beyond, other head dims in four-wave
# workgroups with 64-key blocks.
PEAK_CASES = [  # (rows, S, L, heads, dh): form
    (1, 256, 700, 8, 40),    # 1 x 64
    (2, 2048, 700, 8, 40),   # 2 x 64 x 2 key sets, sixteen waves
    (3, 4096, 700, 8, 40),   # 2 x 64, eight waves
    (2, 2048, 704, 8, 40),   # 2 x 64 x 2 key sets, sixteen waves
    (1, 4000, 1000, 8, 40),  # 2 x 64 x 2 key sets, ragged queries and last key block
    (1, 300, 700, 8, 64),    # 1 x 64
    (2, 2048, 700, 8, 64),   # 2 x 64
    (1, 2100, 700, 8, 80),   # 1 x 64 (264 workgroups of 64 queries)
    (1, 2048, 700, 8, 80),   # 1 x 64 x 2 key sets
    (16, 1024, 700, 8, 80),  # 2 x 64
    (2, 200, 700, 8, 160),   # 1 x 32 x 2 key sets
    (16, 256, 700, 8, 160),  # 2 x 64
    (1, 250, 700, 4, 16),    # 1 x 64
    (8, 1024, 700, 4, 16),   # 2 x 64
]


@pytest.mark.parametrize("kind", ["plant", "hot"])
@pytest.mark.parametrize("rows,S,L,heads,dh", PEAK_CASES)
def test_attention_peaked_scores_take_the_rescale_branch(rows, S, L, heads, dh, kind):
    """scale = 2^-3 / log2(e): the kernel's pre-scaled float16 queries are then
    exact, so large scores carry no query rounding and the float32 oracle is
    the reference at the usual tolerance.  "plant": q, k ~ 2 N(0, 1); for
    queries in several query blocks, a key in key block 2 (of 128; 4 of 64) is
    set to a multiple of the query scoring 9 (log2 units) above everything
    before it, and a second key three blocks later 9 above that, so the
    accumulators hold real mass when the reference moves.  "hot": every query
    scaled by 8, so the reference moves in most blocks."""
    print(f"op attention peaked {kind} rows={rows} S={S} L={L} heads={heads} dh={dh}",
          flush=True)
    C = heads * dh
    rng = np.random.default_rng([S, L, dh, rows, kind == "hot"])
    q = 2.0 * rng.standard_normal((rows, S, C))
    k = 2.0 * rng.standard_normal((rows, L, C))
    v = rng.standard_normal((rows, L, C))
    if kind == "hot":
        q *= 8.0
    q, k, v = (a.astype(np.float16) for a in (q, k, v))
    sc = 0.125  # scores in log2 units: s = q . k / 8
    if kind == "plant":
        for r in range(rows):
            for h in range(heads):
                cols = slice(h * dh, (h + 1) * dh)
                # one query per 64-query workgroup block at a few places, at
                # most one plant per key row (a key row is shared by all queries)
                for n, i in enumerate((5 + 64 * h, S // 2 + h, S - 1 - h)):
                    i %= S
                    qi = q[r, i, cols].astype(np.float64)
                    for step, j in enumerate((263 + 7 * n, 263 + 7 * n + 3 * 128)):
                        j += h % 3
                        before = sc * (k[r, :j, cols].astype(np.float64) @ qi)
                        target = before.max() + 9.0
                        k[r, j, cols] = (qi * (target / (sc * qi @ qi))).astype(np.float16)
    _check(q, k, v, heads, sc / np.log2(np.e), 4e-3)
