"""Seeded synthetic data: cache embeddings, queries, contexts and latents.

Stand-ins for CLIP prompt embeddings (768-d unit vectors, cosine similarity)
and for the prompt stream: no dataset item is reproduced.

Cluster recipe: centres mu_c uniform on the unit sphere; a member is
normalize(mu_c + sigma * g) with g ~ N(0, I_d) (sigma per coordinate).
Rows are generated in fixed chunks of CHUNK rows, each from its own PCG64
stream, so a row's value depends only on (seed, row index).
"""
import numpy as np

CHUNK = 65536


def to_bf16_bits(x):
    """float32 -> uint16 bfloat16 bit patterns, round to nearest even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    # finite inputs cannot overflow: 0xFF7FFFFF + 0x8000 < 2**32
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return u.astype(np.uint16)


def from_bf16_bits(b):
    """uint16 bfloat16 bit patterns -> float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def _into_cone(mu, axis, cone):
    """Unit centres at cosine `cone` to the unit `axis`: cone * axis + sqrt(1 - cone^2)
    times the normalised component of mu orthogonal to the axis."""
    mu = mu - (mu @ axis)[:, None] * axis[None, :]
    mu /= np.linalg.norm(mu, axis=1, keepdims=True)
    return cone * axis[None, :] + np.sqrt(1.0 - cone * cone) * mu


def cluster_centres(clusters, d, seed, cone=0.0):
    """Unit centres, uniform on the sphere; with cone > 0, inside a cone around a
    seeded axis (every centre at cosine `cone` to it), the anisotropy of text-encoder
    embedding spaces, where a linear one-class model can tell in-domain prompts from
    off-domain ones."""
    rng = np.random.default_rng([seed, 0])
    mu = rng.standard_normal((clusters, d))
    mu /= np.linalg.norm(mu, axis=1, keepdims=True)
    if cone > 0.0:
        axis = np.random.default_rng([seed, 9]).standard_normal(d)
        mu = _into_cone(mu, axis / np.linalg.norm(axis), cone)
    return mu.astype(np.float32)


def _chunk_rows(mu, sigma, seed, chunk_index, rows):
    rng = np.random.default_rng([seed, 1, chunk_index])
    cid = rng.integers(0, mu.shape[0], size=rows)
    x = rng.standard_normal((rows, mu.shape[1]), dtype=np.float32)
    x *= np.float32(sigma)
    x += mu[cid]
    nrm = np.sqrt(np.einsum("ij,ij->i", x, x, dtype=np.float32))
    x /= nrm[:, None]
    return x


def make_cache(n, d, clusters, sigma, seed, dtype="bf16", dup_pairs=(), threads=16, cone=0.0):
    """Cache of n unit-norm embeddings.

    dtype "f32" -> float32 [n][d]; "bf16" -> uint16 bit patterns [n][d].
    dup_pairs: (i, j) pairs; row j is overwritten with an exact copy of row i.
    cone: centres inside a cone (cluster_centres).
    Chunks have their own streams, so the values do not depend on `threads`.
    """
    from concurrent.futures import ThreadPoolExecutor
    mu = cluster_centres(clusters, d, seed, cone)
    out = np.empty((n, d), dtype=np.float32 if dtype == "f32" else np.uint16)

    def fill(c):
        start = c * CHUNK
        rows = min(CHUNK, n - start)
        x = _chunk_rows(mu, sigma, seed, c, rows)
        out[start:start + rows] = x if dtype == "f32" else to_bf16_bits(x)

    nchunks = (n + CHUNK - 1) // CHUNK
    if threads > 1 and nchunks > 1:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(fill, range(nchunks)))
    else:
        for c in range(nchunks):
            fill(c)
    for i, j in dup_pairs:
        out[j] = out[i]
    return out


def cache_rows_f32(cache, rows):
    rows = np.asarray(rows)
    sel = cache[rows]
    return sel.astype(np.float32) if sel.dtype == np.float32 else from_bf16_bits(sel)


def make_queries_at_sims(targets, sims, seed):
    """q = s * t_hat + sqrt(1 - s^2) * u, u a random unit vector orthogonal to t_hat.

    targets: float32 [m][d]; sims: length m.  Returns float32 [m][d] unit vectors whose
    cosine with the matching target is s (up to float32 rounding).
    """
    rng = np.random.default_rng([seed, 2])
    t = np.asarray(targets, dtype=np.float64)
    t = t / np.linalg.norm(t, axis=1, keepdims=True)
    g = rng.standard_normal(t.shape)
    g -= np.einsum("ij,ij->i", g, t)[:, None] * t
    g /= np.linalg.norm(g, axis=1, keepdims=True)
    s = np.asarray(sims, dtype=np.float64)[:, None]
    return (s * t + np.sqrt(1.0 - s * s) * g).astype(np.float32)


def make_cluster_queries(m, d, clusters, sigma, cache_seed, seed):
    """Fresh draws from the cache's cluster process (new prompts of a popular theme)."""
    return cluster_queries_from(cluster_centres(clusters, d, cache_seed), m, sigma, seed)


def cluster_queries_from(mu, m, sigma, seed):
    """Fresh draws normalize(mu_c + sigma * g) around given centres mu [clusters][d]."""
    mu = np.asarray(mu, dtype=np.float32)
    clusters, d = mu.shape
    rng = np.random.default_rng([seed, 3])
    cid = rng.integers(0, clusters, size=m)
    x = mu[cid].astype(np.float64) + sigma * rng.standard_normal((m, d))
    return (x / np.linalg.norm(x, axis=1, keepdims=True)).astype(np.float32)


def make_prompt_stream(n, d, seed, p_new=0.35, sims=(0.97, 0.92, 0.87, 0.8, 0.7)):
    """A stream of n request embeddings (float32 unit vectors [n][d]): request j is a
    fresh draw with probability p_new, else a rewording of a uniformly chosen earlier
    request, at a cosine similarity drawn uniformly from sims."""
    rng = np.random.default_rng([seed, 8])
    out = np.empty((n, d), dtype=np.float32)
    for j in range(n):
        g = rng.standard_normal(d)
        if j == 0 or rng.random() < p_new:
            out[j] = g / np.linalg.norm(g)
            continue
        t = out[int(rng.integers(0, j))].astype(np.float64)
        t /= np.linalg.norm(t)
        s = float(sims[int(rng.integers(0, len(sims)))])
        g -= (g @ t) * t
        g /= np.linalg.norm(g)
        out[j] = s * t + np.sqrt(1.0 - s * s) * g
    return out


def make_contexts(b, length, dim, seed):
    """Text-encoder output stand-in: N(0, 1), rounded to bfloat16 values (float32 array)."""
    rng = np.random.default_rng([seed, 4])
    x = rng.standard_normal((b, length, dim), dtype=np.float32)
    return from_bf16_bits(to_bf16_bits(x)).reshape(b, length, dim)


def make_pooled(b, dim, seed):
    """Pooled text-embedding stand-in (SDXL): N(0, 1), rounded to bfloat16 values."""
    rng = np.random.default_rng([seed, 7])
    x = rng.standard_normal((b, dim), dtype=np.float32)
    return from_bf16_bits(to_bf16_bits(x)).reshape(b, dim)


def make_latents(b, c, h, w, seed):
    """x_N ~ N(0, I) in float32 [b][c][h][w]."""
    rng = np.random.default_rng([seed, 5])
    return rng.standard_normal((b, c, h, w), dtype=np.float32)


def make_k_values(b, choices, seed):
    rng = np.random.default_rng([seed, 6])
    return rng.choice(np.asarray(choices, dtype=np.int32), size=b)


def _device_centres(g, clusters, d, device, cone=0.0):
    import torch
    mu = torch.randn(clusters, d, generator=g, device=device, dtype=torch.float32)
    mu = mu / mu.norm(dim=1, keepdim=True)
    if cone > 0.0:  # the axis is the generator's next draw
        axis = torch.randn(d, generator=g, device=device, dtype=torch.float32)
        axis /= axis.norm()
        mu = mu - (mu @ axis)[:, None] * axis[None, :]
        mu /= mu.norm(dim=1, keepdim=True)
        mu = cone * axis[None, :] + float(np.sqrt(1.0 - cone * cone)) * mu
    return mu


def cluster_centres_device(clusters, d, seed, device, cone=0.0):
    """The centres make_cache_device draws first from its generator (float32 [clusters][d])."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return _device_centres(g, clusters, d, device, cone)


def make_cache_device(n, d, clusters, sigma, seed, device, chunk=1 << 20, cone=0.0):
    """The same cluster recipe drawn with torch's seeded generator on `device`, for caches
    too large to generate on the host (10M x 768).  Returns a torch.bfloat16 [n][d]
    tensor (round to nearest even); values depend only on (seed, n, d, clusters, sigma,
    chunk) and the device type."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    mu = _device_centres(g, clusters, d, device, cone)
    out = torch.empty((n, d), dtype=torch.bfloat16, device=device)
    for start in range(0, n, chunk):
        rows = min(chunk, n - start)
        cid = torch.randint(0, clusters, (rows,), generator=g, device=device)
        x = torch.randn(rows, d, generator=g, device=device, dtype=torch.float32)
        x.mul_(sigma).add_(mu[cid])
        x /= x.norm(dim=1, keepdim=True)
        out[start:start + rows] = x.to(torch.bfloat16)
    return out
