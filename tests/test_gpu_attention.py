"""GPU parity of the attention kernel (the UNet's self- and cross-attention,
Sec. 2.1) against the oracle's float32 attention on the same float16-valued
inputs, at the head dims of the configurations (16 tiny, 40 / 80 / 160
SD-1.5, 64 SDXL), the 77-token context with its padded V^T rows, ragged
query / key counts, and each launch form of the 40-dim heads (one query block
per wave; two with 128-key blocks at up to 512 workgroups, as at batch 1 over
4,096 queries; two with 64-key blocks beyond)."""
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
                                               (2, 2048, 333, 8, 40), (3, 4096, 200, 8, 40)])
def test_attention(rows, S, L, heads, dh):
    import paper_2312_04429_amd as P
    print(f"op attention rows={rows} S={S} L={L} heads={heads} dh={dh}", flush=True)
    C = heads * dh
    rng = np.random.default_rng(S + L + dh)
    h = lambda a: a.astype(np.float16)
    q = h(rng.standard_normal((rows, S, C)))
    k = h(rng.standard_normal((rows, L, C)))
    v = h(rng.standard_normal((rows, L, C)))
    Lp = (L + 7) // 8 * 8
    vt = np.zeros((C, rows * Lp), dtype=np.float16)
    for r in range(rows):
        vt[:, r * Lp:r * Lp + L] = v[r].T
    vt[:, :] = np.where(np.arange(rows * Lp)[None, :] % Lp >= L, np.float16(np.nan), vt)  # unused keys
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    got = P.nv_op_attention(t(q), t(k), t(vt), heads, 1.0 / np.sqrt(dh), L=L, vt_row=Lp)
    got = got.float().cpu().numpy()
    for r in range(rows):
        ref = U.attention(q[r].astype(np.float32), k[r].astype(np.float32),
                          v[r].astype(np.float32), heads)
        np.testing.assert_allclose(got[r], ref, rtol=0, atol=4e-3)
