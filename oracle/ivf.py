"""Inverted-file (IVF) approximate search over the cached prompt embeddings
(test infrastructure only).

The paper's vector DB answers nearest-neighbour queries through an approximate
index (HNSW in Qdrant, Sec. 5.3 and Sec. 6); this is the GPU-friendly
counterpart: the rows are partitioned into L lists around unit centroids,
and a query scans only the rows of its nprobe best lists.

Definitions used (each applies to the oracle and the GPU path alike):
  * scores are the canonical ones of the exact lookup: float64 sums of exact
    products, left to right (oracle.lookup.canonical_scores);
  * centroids start as the rows at caller-drawn indices; a Lloyd step
    assigns every row to its best centroid (lowest list on ties), then
    replaces each non-empty list's centroid by the normalised mean of its
    rows: the float64 sum of the rows in ascending row order, divided by the
    square root of the left-to-right sum of its squared components, rounded
    to float32 and, for a bfloat16 cache, on to bfloat16 (nearest even at
    each step); an empty list keeps its centroid;
  * after the last step the rows are assigned once more; list l holds its
    rows in ascending row order (offsets[l] .. offsets[l+1]);
  * a query ranks the lists by its score against their centroids (higher
    first, lower list on ties), takes the first nprobe, and returns the best
    row among them (higher score first, lower row on ties), its score rounded
    to float32 and the selector's K; no probed row: -1, -inf, 0.
"""
import numpy as np

from . import lookup as LK


def _as_f64(rows):
    rows = np.asarray(rows)
    if rows.dtype == np.uint16:
        return (rows.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return rows.astype(np.float64)


def _round_like(v, dtype):
    """float64 -> the cache's storage: float32 (nearest even), then for a bfloat16
    cache its nearest-even bfloat16 bit pattern."""
    f = np.asarray(v, dtype=np.float64).astype(np.float32)
    if dtype != np.uint16:
        return f
    u = f.view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >>
            np.uint32(16)).astype(np.uint16)


def assign(rows, cents):
    """Best centroid per row (canonical scores, lowest list on ties)."""
    out = np.empty(rows.shape[0], np.int64)
    cf = np.asarray(cents)
    for i in range(rows.shape[0]):
        q = _as_f64(rows[i:i + 1])[0].astype(np.float32)
        sc = LK.canonical_scores(q, cf)
        out[i] = LK.top1(sc)[0]
    return out


def lloyd_centroids(rows, lists, cents):
    """One update: normalised fp64 mean of each non-empty list, rounded to the cache type."""
    x = _as_f64(rows)
    new = np.array(cents, copy=True)
    for l in range(cents.shape[0]):
        members = np.nonzero(lists == l)[0]        # ascending row order
        if members.size == 0:
            continue
        s = np.zeros(x.shape[1])
        for r in members:
            s = s + x[r]
        nrm = np.sqrt(float(np.cumsum(s * s)[-1]))
        new[l] = _round_like(s / nrm, cents.dtype)
    return new


def build(rows, init, iters):
    """Centroids, row lists (perm of row ids grouped by list) and list offsets."""
    cents = np.array(rows[np.asarray(init)], copy=True)
    for _ in range(iters):
        cents = lloyd_centroids(rows, assign(rows, cents), cents)
    lists = assign(rows, cents)
    L = cents.shape[0]
    perm = np.concatenate([np.nonzero(lists == l)[0] for l in range(L)]).astype(np.int64)
    offsets = np.zeros(L + 1, np.int64)
    offsets[1:] = np.cumsum(np.bincount(lists, minlength=L))
    return cents, lists, perm, offsets


def search(queries, rows, cents, perm, offsets, nprobe, thresholds, k_values):
    """Returns (idx int64[m], sim float32[m], K int32[m], probed lists [m][nprobe])."""
    queries = np.asarray(queries, dtype=np.float32)
    m, L = queries.shape[0], cents.shape[0]
    idx = np.full(m, -1, np.int64)
    sim = np.full(m, -np.inf, np.float32)
    kk = np.zeros(m, np.int32)
    probed = np.zeros((m, nprobe), np.int64)
    for j in range(m):
        cs = LK.canonical_scores(queries[j], cents)
        order = sorted(range(L), key=lambda l: (-cs[l], l))[:nprobe]
        probed[j] = order
        best, bi = -np.inf, -1
        for l in order:
            members = perm[offsets[l]:offsets[l + 1]]
            if members.size == 0:
                continue
            sc = LK.canonical_scores(queries[j], rows[members])
            for r, v in zip(members, sc):
                if v > best or (v == best and r < bi):
                    best, bi = v, int(r)
        if bi >= 0:
            idx[j] = bi
            sim[j] = np.float32(best)
            kk[j] = LK.select_k(sim[j], thresholds, k_values)
    return idx, sim, kk, probed
