"""Latent-diffusion UNet epsilon predictor in float32 NumPy (test infrastructure only).

Sec. 2.1: the denoiser is a UNet backbone conditioned on the text through
cross-attention, working on a latent.  The paper prints no architecture; the
topology follows the latent-diffusion / Stable-Diffusion layout described by
the workload configuration (channels per level, ResBlocks per level,
transformer depth per level, heads, GroupNorm groups, context shape):

  time embedding : [cos(t f_k), sin(t f_k)], f_k = exp(-ln(1e4) k / (C0/2)),
                   Linear(C0, 4C0) -> SiLU -> Linear(4C0, 4C0) (+ pooled vector)
  ResBlock       : h = conv3x3(SiLU(GN(x))) + Linear(SiLU(temb));
                   h = conv3x3(SiLU(GN(h))); out = skip(x) + h
                   (skip = 1x1 projection when channels change)
  Transformer    : h = proj_in(GN(x)) over tokens; per depth
                   h += SelfAttn(LN(h)); h += CrossAttn(LN(h), ctx);
                   h += W2 (a * GELU_erf(g)) with [a | g] = W1 LN(h) + b1;
                   out = proj_out(h) + x
  attention      : softmax(Q K^T / sqrt(d_head)) V per head, q/k/v without bias
  down / up      : conv3x3 stride 2 / nearest x2 then conv3x3
  skips          : activations saved on the way down, concatenated [h, skip]
                   on the way up, last saved first
  out            : GN -> SiLU -> conv3x3 to the latent channels

One sample at a time, NCHW float32.  Convolutions are im2col + a float32
matrix product (the library primitive); nothing is fused.
"""
import numpy as np
from scipy.special import erf

F32 = np.float32


def silu(x):
    return (x / (F32(1.0) + np.exp(-x))).astype(F32)


def gelu_erf(x):
    return (F32(0.5) * x * (F32(1.0) + erf(x / np.sqrt(F32(2.0))).astype(F32))).astype(F32)


def conv3x3(x, w, b, stride=1):
    """x [C][H][W], w [Co][C][3][3], zero padding 1."""
    c, h, wd = x.shape
    co = w.shape[0]
    ho = (h - 1) // stride + 1
    wo = (wd - 1) // stride + 1
    xp = np.zeros((c, h + 2, wd + 2), dtype=F32)
    xp[:, 1:h + 1, 1:wd + 1] = x
    cols = np.empty((c, 3, 3, ho, wo), dtype=F32)
    for ky in range(3):
        for kx in range(3):
            cols[:, ky, kx] = xp[:, ky:ky + stride * (ho - 1) + 1:stride,
                                 kx:kx + stride * (wo - 1) + 1:stride]
    out = w.reshape(co, c * 9) @ cols.reshape(c * 9, ho * wo)
    return (out + b[:, None]).reshape(co, ho, wo).astype(F32)


def linear(x, w, b=None):
    """x [S][in], w [out][in]."""
    y = x @ w.T
    if b is not None:
        y = y + b
    return y.astype(F32)


def group_norm(x, groups, gamma, beta, eps):
    c = x.shape[0]
    xg = x.reshape(groups, -1)
    mean = xg.mean(axis=1, dtype=F32)[:, None]
    var = ((xg - mean) ** 2).mean(axis=1, dtype=F32)[:, None]
    y = ((xg - mean) / np.sqrt(var + F32(eps))).reshape(x.shape)
    return (y * gamma.reshape(c, 1, 1) + beta.reshape(c, 1, 1)).astype(F32)


def layer_norm(x, gamma, beta, eps):
    mean = x.mean(axis=-1, dtype=F32, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, dtype=F32, keepdims=True)
    return (((x - mean) / np.sqrt(var + F32(eps))) * gamma + beta).astype(F32)


def attention(q, k, v, heads):
    """q [S][C], k, v [L][C] -> [S][C]; fp32 softmax per head."""
    s_len, c = q.shape
    dh = c // heads
    scale = F32(1.0 / np.sqrt(dh))
    out = np.empty((s_len, c), dtype=F32)
    for h in range(heads):
        sl = slice(h * dh, (h + 1) * dh)
        sc = (q[:, sl] @ k[:, sl].T) * scale
        sc = sc - sc.max(axis=1, keepdims=True)
        p = np.exp(sc)
        p = p / p.sum(axis=1, keepdims=True, dtype=F32)
        out[:, sl] = p @ v[:, sl]
    return out


def timestep_embedding(t, dim):
    half = dim // 2
    k = np.arange(half, dtype=F32)
    freqs = np.exp(-np.log(F32(10000.0)) * k / F32(half)).astype(F32)
    arg = F32(t) * freqs
    return np.concatenate([np.cos(arg), np.sin(arg)]).astype(F32)


def upsample_nearest2(x):
    return np.repeat(np.repeat(x, 2, axis=1), 2, axis=2)


class UNet:
    """Epsilon predictor eps(x_t, t, ctx[, pooled]) for one sample."""

    def __init__(self, cfg, weights):
        self.cfg = cfg
        self.w = weights
        self.L = len(cfg["ch"])

    def heads(self, c):
        cfg = self.cfg
        return cfg["n_heads"] if cfg["n_heads"] > 0 else c // cfg["head_dim"]

    def _gn(self, x, name):
        return group_norm(x, self.cfg["gn_groups"], self.w[name + ".g"], self.w[name + ".b"],
                          self.cfg["gn_eps"])

    def _ln(self, x, name):
        return layer_norm(x, self.w[name + ".g"], self.w[name + ".b"], self.cfg["ln_eps"])

    def _conv(self, x, name, stride=1):
        return conv3x3(x, self.w[name + ".w"], self.w[name + ".b"], stride)

    def _lin(self, x, name, bias=True):
        return linear(x, self.w[name + ".w"], self.w[name + ".b"] if bias else None)

    def time_embed(self, t, pooled=None):
        e = timestep_embedding(t, self.cfg["ch"][0])[None, :]
        e = self._lin(silu(self._lin(e, "time.l1")), "time.l2")[0]
        if pooled is not None:
            e = (e + pooled).astype(F32)
        return e

    def resblock(self, x, temb, name):
        h = self._conv(silu(self._gn(x, name + ".gn1")), name + ".conv1")
        tproj = self._lin(silu(temb)[None, :], name + ".temb")[0]
        h = (h + tproj[:, None, None]).astype(F32)
        h = self._conv(silu(self._gn(h, name + ".gn2")), name + ".conv2")
        if name + ".skip.w" in self.w:
            c, hh, ww = x.shape
            sk = self._lin(x.reshape(c, hh * ww).T, name + ".skip").T.reshape(-1, hh, ww)
        else:
            sk = x
        return (sk + h).astype(F32)

    def transformer(self, x, ctx, name, depth):
        c, hh, ww = x.shape
        heads = self.heads(c)
        h = self._gn(x, name + ".gn").reshape(c, hh * ww).T.copy()
        h = self._lin(h, name + ".proj_in")
        for j in range(depth):
            b = f"{name}.blk{j}"
            n1 = self._ln(h, b + ".ln1")
            a = attention(self._lin(n1, b + ".attn1.q", False), self._lin(n1, b + ".attn1.k", False),
                          self._lin(n1, b + ".attn1.v", False), heads)
            h = (h + self._lin(a, b + ".attn1.o")).astype(F32)
            n2 = self._ln(h, b + ".ln2")
            a = attention(self._lin(n2, b + ".attn2.q", False), self._lin(ctx, b + ".attn2.k", False),
                          self._lin(ctx, b + ".attn2.v", False), heads)
            h = (h + self._lin(a, b + ".attn2.o")).astype(F32)
            n3 = self._ln(h, b + ".ln3")
            f = self._lin(n3, b + ".ff1")
            half = f.shape[1] // 2
            g = (f[:, :half] * gelu_erf(f[:, half:])).astype(F32)
            h = (h + self._lin(g, b + ".ff2")).astype(F32)
        h = self._lin(h, name + ".proj_out")
        return (h.T.reshape(c, hh, ww) + x).astype(F32)

    def __call__(self, x, t, ctx, pooled=None):
        cfg = self.cfg
        x = np.asarray(x, dtype=F32)
        ctx = np.asarray(ctx, dtype=F32)
        temb = self.time_embed(t, pooled)
        h = self._conv(x, "conv_in")
        skips = [h]
        for lv in range(self.L):
            for r in range(cfg["n_res"]):
                h = self.resblock(h, temb, f"down{lv}.res{r}")
                if cfg["depth"][lv] > 0:
                    h = self.transformer(h, ctx, f"down{lv}.attn{r}", cfg["depth"][lv])
                skips.append(h)
            if lv < self.L - 1:
                h = self._conv(h, f"down{lv}.ds", stride=2)
                skips.append(h)
        h = self.resblock(h, temb, "mid.res0")
        if cfg["mid_depth"] > 0:
            h = self.transformer(h, ctx, "mid.attn", cfg["mid_depth"])
        h = self.resblock(h, temb, "mid.res1")
        for lv in reversed(range(self.L)):
            for r in range(cfg["n_res"] + 1):
                h = np.concatenate([h, skips.pop()], axis=0)
                h = self.resblock(h, temb, f"up{lv}.res{r}")
                if cfg["depth"][lv] > 0:
                    h = self.transformer(h, ctx, f"up{lv}.attn{r}", cfg["depth"][lv])
            if lv > 0:
                h = self._conv(upsample_nearest2(h), f"up{lv}.us")
        h = silu(self._gn(h, "out.gn"))
        return self._conv(h, "conv_out")


def make_eps_fn(unet, cond, uncond, pooled=None):
    """eps_fn(x, t) -> (eps_uncond, eps_cond) for ddim.denoise, one sample."""
    def fn(x, t):
        return unet(x, t, uncond, pooled), unet(x, t, cond, pooled)
    return fn
