"""Pins of the oracle's UNet layers and topology.

Layer pins use definitions other than the oracle's own code path: direct
convolution loops, float64 library routines from PyTorch-CPU (tests only),
math.erf, and closed forms of the time embedding.  The topology is pinned by
its parameter count against the paper's SD-class SmallModel (about 860 M
parameters, Sec. 7.1) and by an independent float64 PyTorch-functional
composition of the same network on the tiny shape.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as TF

import synth
from oracle import unet as U

F64 = torch.float64


def test_conv3x3_matches_direct_loops():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((3, 5, 6)).astype(np.float32)
    w = rng.standard_normal((2, 3, 3, 3)).astype(np.float32)
    b = rng.standard_normal(2).astype(np.float32)
    for stride in (1, 2):
        got = U.conv3x3(x, w, b, stride)
        ho, wo = (5 - 1) // stride + 1, (6 - 1) // stride + 1
        ref = np.zeros((2, ho, wo))
        for o in range(2):
            for yy in range(ho):
                for xx in range(wo):
                    s = float(b[o])
                    for c in range(3):
                        for ky in range(3):
                            for kx in range(3):
                                iy, ix = yy * stride + ky - 1, xx * stride + kx - 1
                                if 0 <= iy < 5 and 0 <= ix < 6:
                                    s += float(w[o, c, ky, kx]) * float(x[c, iy, ix])
                    ref[o, yy, xx] = s
        np.testing.assert_allclose(got, ref, rtol=1e-5, atol=1e-5)


def test_conv_groupnorm_layernorm_attention_vs_torch_f64():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((16, 7, 9)).astype(np.float32)
    w = (0.1 * rng.standard_normal((8, 16, 3, 3))).astype(np.float32)
    b = rng.standard_normal(8).astype(np.float32)
    ref = TF.conv2d(torch.tensor(x[None], dtype=F64), torch.tensor(w, dtype=F64),
                    torch.tensor(b, dtype=F64), stride=2, padding=1)[0].numpy()
    np.testing.assert_allclose(U.conv3x3(x, w, b, 2), ref, rtol=1e-5, atol=1e-5)

    g = (1 + 0.1 * rng.standard_normal(16)).astype(np.float32)
    be = (0.1 * rng.standard_normal(16)).astype(np.float32)
    ref = TF.group_norm(torch.tensor(x[None], dtype=F64), 4, torch.tensor(g, dtype=F64),
                        torch.tensor(be, dtype=F64), eps=1e-5)[0].numpy()
    np.testing.assert_allclose(U.group_norm(x, 4, g, be, 1e-5), ref, rtol=1e-4, atol=1e-5)

    t = rng.standard_normal((11, 16)).astype(np.float32) * 3 + 1
    ref = TF.layer_norm(torch.tensor(t, dtype=F64), (16,), torch.tensor(g, dtype=F64),
                        torch.tensor(be, dtype=F64), eps=1e-5).numpy()
    np.testing.assert_allclose(U.layer_norm(t, g, be, 1e-5), ref, rtol=1e-4, atol=1e-5)

    q = rng.standard_normal((13, 16)).astype(np.float32)
    k = rng.standard_normal((5, 16)).astype(np.float32)
    v = rng.standard_normal((5, 16)).astype(np.float32)
    tq = torch.tensor(q, dtype=F64).reshape(13, 4, 4).transpose(0, 1)
    tk = torch.tensor(k, dtype=F64).reshape(5, 4, 4).transpose(0, 1)
    tv = torch.tensor(v, dtype=F64).reshape(5, 4, 4).transpose(0, 1)
    ref = TF.scaled_dot_product_attention(tq, tk, tv).transpose(0, 1).reshape(13, 16).numpy()
    np.testing.assert_allclose(U.attention(q, k, v, 4), ref, rtol=1e-5, atol=1e-5)


def test_gelu_silu_pointwise():
    xs = np.linspace(-6, 6, 97).astype(np.float32)
    g = U.gelu_erf(xs)
    s = U.silu(xs)
    for i, v in enumerate(xs.astype(np.float64)):
        assert g[i] == pytest.approx(0.5 * v * (1 + math.erf(v / math.sqrt(2))), rel=1e-5, abs=1e-6)
        assert s[i] == pytest.approx(v / (1 + math.exp(-v)), rel=1e-5, abs=1e-6)


def test_time_embedding_closed_form():
    e0 = U.timestep_embedding(0, 32)
    np.testing.assert_array_equal(e0[:16], np.ones(16, np.float32))
    np.testing.assert_array_equal(e0[16:], np.zeros(16, np.float32))
    e = U.timestep_embedding(981, 320)
    assert e[0] == pytest.approx(math.cos(981.0), abs=1e-4)      # f_0 = 1
    assert e[160] == pytest.approx(math.sin(981.0), abs=1e-4)
    k = 37
    f = math.exp(-math.log(1e4) * k / 160)
    assert e[k] == pytest.approx(math.cos(981.0 * f), abs=1e-4)
    assert e[160 + k] == pytest.approx(math.sin(981.0 * f), abs=1e-4)


def test_sd15_parameter_count_matches_paper_smallmodel():
    """(C-P7) the SD-1.5 topology has 859 520 964 parameters; the paper's SD-class
    SmallModel has about 860 M (Sec. 7.1)."""
    n = synth.param_count(synth.unet_config("sd15"))
    assert n == 859_520_964
    assert abs(n - 860e6) / 860e6 < 1e-3


# ---- independent float64 composition with torch.nn.functional (tests only) ----

def _t(a):
    return torch.tensor(np.asarray(a), dtype=F64)


def _torch_unet(cfg, w, x, t, ctx, pooled=None):
    W = {k: _t(v) for k, v in w.items()}
    G, eg, el = cfg["gn_groups"], cfg["gn_eps"], cfg["ln_eps"]
    c0 = cfg["ch"][0]
    half = c0 // 2
    fr = torch.exp(-math.log(10000.0) * torch.arange(half, dtype=F64) / half)
    temb = torch.cat([torch.cos(t * fr), torch.sin(t * fr)])
    temb = TF.linear(TF.silu(TF.linear(temb, W["time.l1.w"], W["time.l1.b"])), W["time.l2.w"],
                     W["time.l2.b"])
    if pooled is not None:  # added as is to the embedding, before the ResBlocks' SiLU
        temb = temb + _t(pooled)
    c_ = _t(ctx)

    def conv(h, n, stride=1):
        return TF.conv2d(h, W[n + ".w"], W[n + ".b"], stride=stride, padding=1)

    def gn(h, n):
        return TF.group_norm(h, G, W[n + ".g"], W[n + ".b"], eps=eg)

    def res(h, n):
        y = conv(TF.silu(gn(h, n + ".gn1")), n + ".conv1")
        y = y + TF.linear(TF.silu(temb), W[n + ".temb.w"], W[n + ".temb.b"])[None, :, None, None]
        y = conv(TF.silu(gn(y, n + ".gn2")), n + ".conv2")
        if n + ".skip.w" in W:
            h = TF.conv2d(h, W[n + ".skip.w"][:, :, None, None], W[n + ".skip.b"])
        return h + y

    def attn(q, k, v, heads):
        s, c = q.shape
        dh = c // heads
        f = lambda z: z.reshape(z.shape[0], heads, dh).transpose(0, 1)
        return TF.scaled_dot_product_attention(f(q), f(k), f(v)).transpose(0, 1).reshape(s, c)

    def tr(h, n, depth):
        _, c, hh, ww = h.shape
        heads = cfg["n_heads"] if cfg["n_heads"] > 0 else c // cfg["head_dim"]
        y = gn(h, n + ".gn")[0].reshape(c, -1).T
        y = TF.linear(y, W[n + ".proj_in.w"], W[n + ".proj_in.b"])
        for j in range(depth):
            b = f"{n}.blk{j}"
            ln = lambda z, m: TF.layer_norm(z, (c,), W[m + ".g"], W[m + ".b"], eps=el)
            z = ln(y, b + ".ln1")
            y = y + TF.linear(attn(z @ W[b + ".attn1.q.w"].T, z @ W[b + ".attn1.k.w"].T,
                                   z @ W[b + ".attn1.v.w"].T, heads), W[b + ".attn1.o.w"],
                              W[b + ".attn1.o.b"])
            z = ln(y, b + ".ln2")
            y = y + TF.linear(attn(z @ W[b + ".attn2.q.w"].T, c_ @ W[b + ".attn2.k.w"].T,
                                   c_ @ W[b + ".attn2.v.w"].T, heads), W[b + ".attn2.o.w"],
                              W[b + ".attn2.o.b"])
            z = ln(y, b + ".ln3")
            a, g = TF.linear(z, W[b + ".ff1.w"], W[b + ".ff1.b"]).chunk(2, dim=-1)
            y = y + TF.linear(a * TF.gelu(g), W[b + ".ff2.w"], W[b + ".ff2.b"])
        y = TF.linear(y, W[n + ".proj_out.w"], W[n + ".proj_out.b"])
        return y.T.reshape(1, c, hh, ww) + h

    L = len(cfg["ch"])
    h = conv(_t(x)[None], "conv_in")
    sk = [h]
    for lv in range(L):
        for r in range(cfg["n_res"]):
            h = res(h, f"down{lv}.res{r}")
            if cfg["depth"][lv]:
                h = tr(h, f"down{lv}.attn{r}", cfg["depth"][lv])
            sk.append(h)
        if lv < L - 1:
            h = conv(h, f"down{lv}.ds", 2)
            sk.append(h)
    h = res(h, "mid.res0")
    if cfg["mid_depth"]:
        h = tr(h, "mid.attn", cfg["mid_depth"])
    h = res(h, "mid.res1")
    for lv in reversed(range(L)):
        for r in range(cfg["n_res"] + 1):
            h = res(torch.cat([h, sk.pop()], dim=1), f"up{lv}.res{r}")
            if cfg["depth"][lv]:
                h = tr(h, f"up{lv}.attn{r}", cfg["depth"][lv])
        if lv > 0:
            h = conv(TF.interpolate(h, scale_factor=2, mode="nearest"), f"up{lv}.us")
    h = conv(TF.silu(gn(h, "out.gn")), "conv_out")
    return h[0].numpy()


@pytest.mark.parametrize("over", [{}, dict(n_res=2, mid_depth=0, depth=(1, 2))])
def test_tiny_unet_matches_independent_torch_composition(over):
    cfg = synth.unet_config("tiny", **over)
    w = synth.make_weights(cfg, 0)
    x = synth.make_latents(1, 4, cfg["H"], cfg["W"], 2000)[0]
    ctx = synth.make_contexts(1, cfg["ctx_len"], cfg["ctx_dim"], 3)[0]
    got = U.UNet(cfg, w)(x, 741, ctx)
    ref = _torch_unet(cfg, w, x, 741.0, ctx)
    np.testing.assert_allclose(got, ref, rtol=1e-3, atol=2e-4)


def test_sdxl_topology_with_pooled_vector_matches_independent_torch_composition():
    """The SDXL-shaped rules on a narrow network: head count from head_dim (1, 2
    and 4 heads of 64), transformer depth 0/2 per level and a depth-10 middle
    block, and a pooled vector as wide as the time embedding added to it.  A
    pooled vector added before time.l2 or after the ResBlocks' SiLU, a head
    count taken from n_heads, or a dropped depth block fails the comparison."""
    cfg = synth.unet_config("sdxl", H=8, W=8, ch=(64, 128, 256), ctx_len=6, ctx_dim=96,
                            pooled_dim=256, depth=(0, 2, 2), mid_depth=10)
    w = synth.make_weights(cfg, 0)
    x = synth.make_latents(1, 4, cfg["H"], cfg["W"], 2002)[0]
    ctx = synth.make_contexts(1, cfg["ctx_len"], cfg["ctx_dim"], 7)[0]
    pooled = synth.make_pooled(1, cfg["pooled_dim"], 8)[0]
    net = U.UNet(cfg, w)
    got = net(x, 601, ctx, pooled)
    ref = _torch_unet(cfg, w, x, 601.0, ctx, pooled)
    np.testing.assert_allclose(got, ref, rtol=1e-3, atol=2e-4)
    # the pooled vector reaches eps (its effect is far above the tolerance)
    plain = _torch_unet(cfg, w, x, 601.0, ctx, None)
    assert np.abs(ref - plain).max() > 50 * 2e-4


def test_context_token_permutation_invariance():
    """Cross-attention pools over context tokens, so permuting them leaves eps unchanged."""
    cfg = synth.unet_config("tiny")
    w = synth.make_weights(cfg, 0)
    x = synth.make_latents(1, 4, 16, 16, 2001)[0]
    ctx = synth.make_contexts(1, 8, 64, 5)[0]
    net = U.UNet(cfg, w)
    perm = np.random.default_rng(3).permutation(8)
    np.testing.assert_allclose(net(x, 501, ctx), net(x, 501, ctx[perm]), rtol=1e-4, atol=1e-5)
