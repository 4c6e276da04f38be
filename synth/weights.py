"""Parameter enumeration and seeded random-init weights for the UNet topologies.

The enumeration order below is the canonical packing order of the weight blob
(conv weights [Cout][Cin][3][3], linear weights [out][in], both row-major).
Values are drawn per tensor from numpy's PCG64 seeded with (seed, tensor
index) and then rounded to bfloat16, so every consumer sees identical values:
  matrices and biases  ~ N(0, 0.02)
  norm scales          ~ 1 + N(0, 0.02)
  norm shifts          ~ N(0, 0.02)
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np

STD = 0.02


def bf16_round(x):
    """Round float32 values to the nearest bfloat16 (ties to even), kept as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    # finite inputs cannot overflow: 0xFF7FFFFF + 0x8000 < 2**32
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return u.view(np.float32)


def param_specs(cfg):
    """List of (name, shape, kind) in canonical order; kind in mat|bias|gamma|beta."""
    specs = []
    c0 = cfg["ch"][0]
    td = 4 * c0
    L = len(cfg["ch"])

    def lin(name, out, inp, bias=True):
        specs.append((name + ".w", (out, inp), "mat"))
        if bias:
            specs.append((name + ".b", (out,), "bias"))

    def conv(name, out, inp, k=3):
        specs.append((name + ".w", (out, inp, k, k), "mat"))
        specs.append((name + ".b", (out,), "bias"))

    def norm(name, c):
        specs.append((name + ".g", (c,), "gamma"))
        specs.append((name + ".b", (c,), "beta"))

    def res(name, cin, cout):
        norm(name + ".gn1", cin)
        conv(name + ".conv1", cout, cin)
        lin(name + ".temb", cout, td)
        norm(name + ".gn2", cout)
        conv(name + ".conv2", cout, cout)
        if cin != cout:
            lin(name + ".skip", cout, cin)

    def transformer(name, c, depth):
        norm(name + ".gn", c)
        lin(name + ".proj_in", c, c)
        for j in range(depth):
            b = f"{name}.blk{j}"
            norm(b + ".ln1", c)
            lin(b + ".attn1.q", c, c, bias=False)
            lin(b + ".attn1.k", c, c, bias=False)
            lin(b + ".attn1.v", c, c, bias=False)
            lin(b + ".attn1.o", c, c)
            norm(b + ".ln2", c)
            lin(b + ".attn2.q", c, c, bias=False)
            lin(b + ".attn2.k", c, cfg["ctx_dim"], bias=False)
            lin(b + ".attn2.v", c, cfg["ctx_dim"], bias=False)
            lin(b + ".attn2.o", c, c)
            norm(b + ".ln3", c)
            lin(b + ".ff1", 8 * c, c)
            lin(b + ".ff2", c, 4 * c)
        lin(name + ".proj_out", c, c)

    lin("time.l1", td, c0)
    lin("time.l2", td, td)
    conv("conv_in", c0, cfg["in_ch"])
    skips = [c0]
    cur = c0
    for lv in range(L):
        cout = cfg["ch"][lv]
        for r in range(cfg["n_res"]):
            res(f"down{lv}.res{r}", cur, cout)
            cur = cout
            if cfg["depth"][lv] > 0:
                transformer(f"down{lv}.attn{r}", cur, cfg["depth"][lv])
            skips.append(cur)
        if lv < L - 1:
            conv(f"down{lv}.ds", cur, cur)
            skips.append(cur)
    res("mid.res0", cur, cur)
    if cfg["mid_depth"] > 0:
        transformer("mid.attn", cur, cfg["mid_depth"])
    res("mid.res1", cur, cur)
    for lv in reversed(range(L)):
        cout = cfg["ch"][lv]
        for r in range(cfg["n_res"] + 1):
            sk = skips.pop()
            res(f"up{lv}.res{r}", cur + sk, cout)
            cur = cout
            if cfg["depth"][lv] > 0:
                transformer(f"up{lv}.attn{r}", cur, cfg["depth"][lv])
        if lv > 0:
            conv(f"up{lv}.us", cur, cur)
    assert not skips
    norm("out.gn", cur)
    conv("conv_out", cfg["out_ch"], cur)
    return specs


def param_count(cfg):
    return int(sum(int(np.prod(s)) for _, s, _ in param_specs(cfg)))


def _one(seed, i, shape, kind, round_bf16):
    rng = np.random.default_rng([seed, i])
    g = rng.standard_normal(shape, dtype=np.float32)
    g *= np.float32(STD)
    if kind == "gamma":
        g += np.float32(1.0)
    return bf16_round(g) if round_bf16 else g


def make_weights(cfg, seed=0, round_bf16=True, threads=8):
    """Return an ordered dict name -> float32 array (bf16-representable values).

    Each tensor has its own stream, so the values do not depend on `threads`.
    """
    specs = param_specs(cfg)
    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        futs = [ex.submit(_one, seed, i, shape, kind, round_bf16)
                for i, (_, shape, kind) in enumerate(specs)]
        return {name: f.result() for (name, _, _), f in zip(specs, futs)}
