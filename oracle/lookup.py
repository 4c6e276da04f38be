"""Cache lookup and cache selector (test infrastructure only).

Follows Sec. 4.3 (Alg. 1: search the vector DB for the closest cached prompt,
then map its score to K) and Sec. 5.3.1 (the cache selector: the first
threshold the similarity strictly exceeds gives K, else K = 0 and the request
falls back to full generation).

Definitions used (readings of the paper):
  * similarity is the inner product of the stored vectors (cosine for the
    unit-norm embeddings of the workloads); no renormalisation;
  * the canonical score of entry i is the float64 sum of q_k * c_ik taken
    strictly left to right over k.  Each product of a float32 (or bfloat16)
    pair is exact in float64, so this value is reproducible anywhere;
  * the best entry is the lowest index among those with the maximal canonical
    score; its similarity is that score rounded to float32;
  * the selector compares that float32 similarity with each float32
    threshold using strict '>', in table order;
  * an empty cache returns index -1, similarity -inf and K = 0.
"""
import numpy as np

ROWS_PER_CHUNK = 16384


def _rows_f32(cache, start, stop):
    blk = cache[start:stop]
    if blk.dtype == np.uint16:  # bfloat16 bit patterns
        return (blk.astype(np.uint32) << 16).view(np.float32)
    return np.asarray(blk, dtype=np.float32)


def canonical_scores(query, cache):
    """float64 score of every cache row for one float32 query, left-to-right sums.

    cache: float32 [n][d] or uint16 bfloat16 bits [n][d].
    """
    q = np.asarray(query, dtype=np.float32).astype(np.float64)
    n, d = cache.shape
    out = np.empty(n, dtype=np.float64)
    for start in range(0, n, ROWS_PER_CHUNK):
        stop = min(n, start + ROWS_PER_CHUNK)
        ct = _rows_f32(cache, start, stop).astype(np.float64).T.copy()  # [d][rows]
        s = np.zeros(stop - start, dtype=np.float64)
        for k in range(d):
            s += ct[k] * q[k]          # exact product, one rounding per addition
        out[start:stop] = s
    return out


def canonical_score_rows(query, cache, rows):
    """Canonical scores of selected rows only (for sampled checks on huge caches)."""
    rows = np.asarray(rows, dtype=np.int64)
    sub = cache[rows]
    return canonical_scores(query, sub)


def select_k(sim, thresholds, k_values):
    """Cache selector: K of the first threshold that sim (float32) strictly exceeds."""
    s = np.float32(sim)
    for thr, k in zip(thresholds, k_values):
        if s > np.float32(thr):
            return int(k)
    return 0


def top1(scores):
    """(index, float64 score) of the maximum, lowest index among ties."""
    best = -np.inf
    idx = -1
    for i, v in enumerate(scores):  # explicit scan: first occurrence wins
        if v > best:
            best, idx = v, i
    return idx, best


def top1_fast(scores):
    """Same result as top1 (np.argmax returns the first maximal index)."""
    if scores.size == 0:
        return -1, -np.inf
    i = int(np.argmax(scores))
    return i, float(scores[i])


def lookup(queries, cache, thresholds, k_values):
    """Returns (idx int64[m], sim float32[m], K int32[m])."""
    queries = np.asarray(queries, dtype=np.float32)
    m = queries.shape[0]
    idx = np.full(m, -1, dtype=np.int64)
    sim = np.full(m, -np.inf, dtype=np.float32)
    kk = np.zeros(m, dtype=np.int32)
    if cache.shape[0] == 0:
        return idx, sim, kk
    for j in range(m):
        sc = canonical_scores(queries[j], cache)
        i, v = top1_fast(sc)
        idx[j] = i
        sim[j] = np.float32(v)
        kk[j] = select_k(sim[j], thresholds, k_values)
    return idx, sim, kk
