"""Python entry points with the C ABI's names (argument marshalling only).

Tensors are torch device tensors; outputs and workspaces are allocated with
torch; every computation happens in libnv.so on the current HIP stream.
"""
import ctypes as C

import numpy as np
import torch

from . import _native as N  # noqa: N812

BF16_DTYPES = (torch.bfloat16, torch.int16, torch.uint16)


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _p(t):
    return C.c_void_p(t.data_ptr()) if t is not None else None


def _need_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("device tensor expected")


def workspace(nbytes, device):
    """A 256-byte aligned device byte buffer: (owner tensor, aligned address)."""
    t = torch.empty(int(nbytes) + 256, dtype=torch.uint8, device=device)
    addr = t.data_ptr()
    return t, addr + (-addr) % 256


def nv_cache_lookup_workspace(m, n, d):
    return int(N.lib.nv_cache_lookup_workspace(m, n, d))


def nv_cache_lookup(queries, cache, thresholds, k_values, ws=None):
    """Exact cosine top-1 + cache selector.  Returns (idx int64, sim f32, K int32) on device."""
    _need_cuda(queries, cache)
    assert queries.dtype == torch.float32 and queries.is_contiguous()
    assert cache.is_contiguous()
    m, d = queries.shape
    n = cache.shape[0]
    if cache.dtype == torch.float32:
        cdt = N.NV_F32
    elif cache.dtype in BF16_DTYPES:
        cdt = N.NV_BF16
    else:
        raise ValueError("cache must be float32 or bfloat16 (bits)")
    thr = (C.c_float * len(thresholds))(*thresholds)
    kv = (C.c_int32 * len(k_values))(*k_values)
    dev = queries.device
    idx = torch.empty(m, dtype=torch.int64, device=dev)
    sim = torch.empty(m, dtype=torch.float32, device=dev)
    kk = torch.empty(m, dtype=torch.int32, device=dev)
    need = nv_cache_lookup_workspace(m, n, d)
    if ws is None:
        _own, addr = workspace(need, dev)
        wbytes = need
    else:
        _own, addr, wbytes = ws
    st = N.lib.nv_cache_lookup(_p(queries), m, _p(cache) if n > 0 else None, cdt, n, d, thr, kv,
                               len(thresholds), _p(idx), _p(sim), _p(kk), C.c_void_p(addr),
                               wbytes, _stream())
    N.check(st, "nv_cache_lookup")
    return idx, sim, kk


def nv_cache_lookup_static(queries, cache, thresholds, k_values, out=None):
    """nv_cache_lookup on the library's own scratch (no workspace, no allocation by
    the library).  out: optional (idx, sim, K) device tensors of m entries to fill."""
    _need_cuda(queries, cache)
    assert queries.dtype == torch.float32 and queries.is_contiguous()
    assert cache.is_contiguous()
    m, d = queries.shape
    n = cache.shape[0]
    if cache.dtype == torch.float32:
        cdt = N.NV_F32
    elif cache.dtype in BF16_DTYPES:
        cdt = N.NV_BF16
    else:
        raise ValueError("cache must be float32 or bfloat16 (bits)")
    thr = (C.c_float * len(thresholds))(*thresholds)
    kv = (C.c_int32 * len(k_values))(*k_values)
    dev = queries.device
    if out is None:
        out = (torch.empty(m, dtype=torch.int64, device=dev),
               torch.empty(m, dtype=torch.float32, device=dev),
               torch.empty(m, dtype=torch.int32, device=dev))
    idx, sim, kk = out
    st = N.lib.nv_cache_lookup_static(_p(queries), m, _p(cache) if n > 0 else None, cdt, n, d,
                                      thr, kv, len(thresholds), _p(idx), _p(sim), _p(kk),
                                      _stream())
    N.check(st, "nv_cache_lookup_static")
    return idx, sim, kk


def nv_gather_states(store, slot_k, payload, n_rows, idx, k, noise, out=None):
    """store [n_store][n_slots][*latent] f32; returns out [B][*latent]; k rewritten in place."""
    _need_cuda(store, idx, k, noise)
    B = idx.shape[0]
    lat = int(np.prod(noise.shape[1:]))
    if out is None:
        out = torch.empty_like(noise)
    sk = (C.c_int32 * len(slot_k))(*slot_k)
    st = N.lib.nv_gather_states(_p(store), store.shape[0], len(slot_k), sk, _p(payload), n_rows,
                                _p(idx), _p(k), _p(noise), B, lat, _p(out), _stream())
    N.check(st, "nv_gather_states")
    return out


def nv_gather_pool(pool, table, slot_k, payload, n_rows, idx, k, noise, out=None):
    """Hole-aware fetch from a state pool: pool [n_pool][*latent] f32, table int32
    [n_entries][n_slots]; returns out [B][*latent]; k becomes the K served (0: noise)."""
    _need_cuda(pool, table, idx, k, noise, payload)
    B = idx.shape[0]
    lat = int(np.prod(noise.shape[1:]))
    if table.dim() != 2 or table.shape[1] != len(slot_k) or table.dtype != torch.int32:
        raise ValueError("table must be int32 [n_entries][len(slot_k)]")
    if pool.dtype != torch.float32 or int(np.prod(pool.shape[1:])) != lat:
        raise ValueError("pool must be float32 [n_pool][*latent]")
    if k.shape[0] != B or noise.shape[0] != B or idx.dtype != torch.int64:
        raise ValueError("idx (int64), k and noise need B rows")
    if payload is not None and payload.shape[0] < n_rows:
        raise ValueError("payload shorter than n_rows")
    if out is None:
        out = torch.empty_like(noise)
    sk = (C.c_int32 * len(slot_k))(*[int(v) for v in slot_k])
    st = N.lib.nv_gather_pool(_p(pool), pool.shape[0], _p(table), table.shape[0], len(slot_k), sk,
                              _p(payload), int(n_rows), _p(idx), _p(k), _p(noise), B, lat,
                              _p(out), _stream())
    N.check(st, "nv_gather_pool")
    return out


def nv_table_update(table, rec):
    """table int32 [n_entries][n_slots]; rec int32 [u][1 + n_slots] (device)."""
    _need_cuda(table, rec)
    assert table.dtype == torch.int32 and rec.dtype == torch.int32 and rec.is_contiguous()
    if rec.dim() != 2 or rec.shape[1] != 1 + table.shape[1]:
        raise ValueError("rec must be [u][1 + n_slots]")
    u = rec.shape[0]
    st = N.lib.nv_table_update(_p(table), table.shape[0], table.shape[1], _p(rec) if u else None,
                               u, _stream())
    N.check(st, "nv_table_update")


def nv_cache_move_rows(cache, n, payload, src, dst):
    """Move cache rows src[i] -> dst[i] (int64 device) and their payload entries."""
    _need_cuda(cache, payload, src, dst)
    count = src.shape[0]
    if dst.shape[0] != count or src.dtype != torch.int64 or dst.dtype != torch.int64:
        raise ValueError("src and dst must be int64 of one length")
    if int(n) > cache.shape[0] or (payload is not None and payload.shape[0] < int(n)):
        raise ValueError("n exceeds the cache or payload rows")
    cdt = N.NV_F32 if cache.dtype == torch.float32 else N.NV_BF16
    st = N.lib.nv_cache_move_rows(_p(cache), cdt, int(n), cache.shape[1], _p(payload),
                                  _p(src) if count else None, _p(dst) if count else None, count,
                                  _stream())
    N.check(st, "nv_cache_move_rows")


class NvIVF:
    """IVF index over a device cache (f32, or bf16 as torch.bfloat16 / int16 bits):
    centroids, row lists and the rows in list order, built on the device."""

    def __init__(self, cache, init, iters=0):
        _need_cuda(cache)
        assert cache.is_contiguous() and cache.dim() == 2
        n, d = cache.shape
        self.dtype = N.NV_F32 if cache.dtype == torch.float32 else N.NV_BF16
        if self.dtype == N.NV_BF16 and cache.dtype not in BF16_DTYPES:
            raise ValueError("cache must be float32 or bfloat16 (bits)")
        init = np.ascontiguousarray(init, dtype=np.int64)
        L = len(init)
        dev = cache.device
        self.n, self.d, self.L = n, d, L
        self.cents = torch.empty((L, d), dtype=cache.dtype, device=dev)
        self.lists = torch.empty(n, dtype=torch.int64, device=dev)
        self.perm = torch.empty(n, dtype=torch.int64, device=dev)
        self.offsets = torch.empty(L + 1, dtype=torch.int64, device=dev)
        self.rows = torch.empty_like(cache)
        need = int(N.lib.nv_ivf_build_workspace(n, d, L))
        own, addr = workspace(need, dev)
        mx = C.c_int64()
        st = N.lib.nv_ivf_build(_p(cache), self.dtype, n, d, init.ctypes.data, L, int(iters),
                                _p(self.cents), _p(self.lists), _p(self.perm), _p(self.offsets),
                                _p(self.rows), C.byref(mx), C.c_void_p(addr), need, _stream())
        N.check(st, "nv_ivf_build")
        del own
        self.max_list = mx.value

    def search(self, queries, nprobe, thresholds, k_values, probed=False):
        """(idx int64, sim f32, K int32[, probed lists int32 [m][nprobe]]) on device."""
        _need_cuda(queries)
        assert queries.dtype == torch.float32 and queries.is_contiguous()
        m = queries.shape[0]
        dev = queries.device
        idx = torch.empty(m, dtype=torch.int64, device=dev)
        sim = torch.empty(m, dtype=torch.float32, device=dev)
        kk = torch.empty(m, dtype=torch.int32, device=dev)
        pr = torch.empty((m, nprobe), dtype=torch.int32, device=dev) if probed else None
        thr = (C.c_float * len(thresholds))(*thresholds)
        kv = (C.c_int32 * len(k_values))(*k_values)
        need = int(N.lib.nv_ivf_search_workspace(m, self.L, nprobe, self.max_list))
        own, addr = workspace(need, dev)
        st = N.lib.nv_ivf_search(_p(queries), m, self.d, _p(self.cents), self.L, _p(self.rows),
                                 self.dtype, _p(self.perm), _p(self.offsets), self.max_list,
                                 int(nprobe), thr, kv, len(thresholds), _p(idx), _p(sim), _p(kk),
                                 _p(pr), C.c_void_p(addr), need, _stream())
        N.check(st, "nv_ivf_search")
        return (idx, sim, kk, pr) if probed else (idx, sim, kk)


def nv_ocsvm_train(rows, nu, order, eta0=1.0):
    """Train the match predictor on host rows (numpy float32, or uint16 bfloat16 bits
    [n][d]) in the visiting order (host int64 [T]).  Returns (w float64 [d], rho)."""
    rows = np.ascontiguousarray(rows)
    cdt = N.NV_BF16 if rows.dtype in (np.uint16, np.int16) else N.NV_F32
    if cdt == N.NV_F32 and rows.dtype != np.float32:
        raise ValueError("rows must be float32 or bfloat16 bits")
    order = np.ascontiguousarray(order, dtype=np.int64)
    n, d = rows.shape
    w = np.empty(d, np.float64)
    rho = C.c_double()
    st = N.lib.nv_ocsvm_train(rows.ctypes.data, cdt, n, d, float(nu), float(eta0),
                              order.ctypes.data, len(order), w.ctypes.data, C.byref(rho))
    N.check(st, "nv_ocsvm_train")
    return w, rho.value


def nv_match_gate(queries, w, rho, tau=0.0, idx=None, sim=None, k=None, score=True):
    """Decision values w.q - rho of the queries (float64 device [m]) and, when a
    lookup's (idx, sim, k) are given, 'no match' for every query below tau."""
    _need_cuda(queries, w, idx, sim, k)
    assert queries.dtype == torch.float32 and queries.is_contiguous()
    assert w.dtype == torch.float64 and w.numel() == queries.shape[1]
    m, d = queries.shape
    out = torch.empty(m, dtype=torch.float64, device=queries.device) if score else None
    st = N.lib.nv_match_gate(_p(queries), m, d, _p(w), float(rho), float(tau), _p(out),
                             _p(idx), _p(sim), _p(k), _stream())
    N.check(st, "nv_match_gate")
    return out


def nv_cache_lookup_gated(queries, cache, thresholds, k_values, w, rho, tau=0.0, ws=None):
    """The lookup with the match predictor in front (Alg. 1): only queries with
    w.q - rho >= tau are searched.  Returns (idx, sim, K, score) on the device and
    the number of queries searched."""
    _need_cuda(queries, cache, w)
    assert queries.dtype == torch.float32 and queries.is_contiguous() and cache.is_contiguous()
    assert w.dtype == torch.float64 and w.numel() == queries.shape[1]
    m, d = queries.shape
    n = cache.shape[0]
    if cache.dtype == torch.float32:
        cdt = N.NV_F32
    elif cache.dtype in BF16_DTYPES:
        cdt = N.NV_BF16
    else:
        raise ValueError("cache must be float32 or bfloat16 (bits)")
    thr = (C.c_float * len(thresholds))(*thresholds)
    kv = (C.c_int32 * len(k_values))(*k_values)
    dev = queries.device
    idx = torch.empty(m, dtype=torch.int64, device=dev)
    sim = torch.empty(m, dtype=torch.float32, device=dev)
    kk = torch.empty(m, dtype=torch.int32, device=dev)
    score = torch.empty(m, dtype=torch.float64, device=dev)
    need = int(N.lib.nv_cache_lookup_gated_workspace(m, n, d))
    if ws is None:
        _own, addr = workspace(need, dev)
        wbytes = need
    else:
        _own, addr, wbytes = ws
    searched = C.c_int32()
    st = N.lib.nv_cache_lookup_gated(_p(queries), m, _p(cache) if n > 0 else None, cdt, n, d, thr,
                                     kv, len(thresholds), _p(w), float(rho), float(tau), _p(idx),
                                     _p(sim), _p(kk), _p(score), C.byref(searched),
                                     C.c_void_p(addr), wbytes, _stream())
    N.check(st, "nv_cache_lookup_gated")
    return idx, sim, kk, score, searched.value


def nv_cache_lookup_gated_workspace(m, n, d):
    return int(N.lib.nv_cache_lookup_gated_workspace(m, n, d))


class NvLCBFU:
    """Host LCBFU maintainer (native); arrays in and out are host numpy arrays."""

    def __init__(self, slot_k, state_capacity, entry_capacity):
        self.slot_k = [int(v) for v in slot_k]
        self.S = len(self.slot_k)
        self.cap, self.ecap = int(state_capacity), int(entry_capacity)
        h = C.c_void_p()
        sk = (C.c_int32 * self.S)(*self.slot_k)
        N.check(N.lib.nv_lcbfu_create(self.S, sk, self.cap, self.ecap, C.byref(h)),
                "nv_lcbfu_create")
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            N.lib.nv_lcbfu_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def access(self, rows, ks):
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        ks = np.ascontiguousarray(ks, dtype=np.int32)
        st = N.lib.nv_lcbfu_access(self._h, len(rows), rows.ctypes.data, ks.ctypes.data)
        N.check(st, "nv_lcbfu_access")

    def insert(self, m):
        S = self.S
        ent = np.empty(m, np.int32)
        pools = np.empty((m, S), np.int32)
        src = np.empty(m * S, np.int64)
        dst = np.empty(m * S, np.int64)
        upd = np.empty((m * S + m, 1 + S), np.int32)
        nm, nu, kept = C.c_int32(), C.c_int32(), C.c_int64()
        st = N.lib.nv_lcbfu_insert(self._h, int(m), ent.ctypes.data, pools.ctypes.data,
                                   src.ctypes.data, dst.ctypes.data, C.byref(nm),
                                   upd.ctypes.data, C.byref(nu), C.byref(kept))
        N.check(st, "nv_lcbfu_insert")
        return {"entries": ent, "pools": pools, "move_src": src[:nm.value],
                "move_dst": dst[:nm.value], "upd": upd[:nu.value], "kept": kept.value}

    def info(self):
        out = np.zeros(5, np.int64)
        N.check(N.lib.nv_lcbfu_info(self._h, out.ctypes.data), "nv_lcbfu_info")
        return dict(zip(("rows", "states", "evicted", "dropped", "stored"), out.tolist()))

    def export(self):
        table = np.empty((self.ecap, self.S), np.int32)
        rows = np.empty(self.info()["rows"], np.int32)
        counts = np.empty(self.cap, np.int64)
        st = N.lib.nv_lcbfu_export(self._h, table.ctypes.data, rows.ctypes.data,
                                   counts.ctypes.data)
        N.check(st, "nv_lcbfu_export")
        return table, rows, counts


def nv_unet_param_count(cfg):
    c = N.make_config(cfg)
    return int(N.lib.nv_unet_param_count(C.byref(c)))


def nv_unet_param_info(cfg, i):
    c = N.make_config(cfg)
    buf = C.create_string_buffer(256)
    n = C.c_int64()
    N.check(N.lib.nv_unet_param_info(C.byref(c), i, buf, 256, C.byref(n)), "nv_unet_param_info")
    return buf.value.decode(), int(n.value)


class NvUNet:
    """Handle of a device-resident UNet (nv_unet_create / nv_unet_destroy)."""

    def __init__(self, cfg, weights):
        self.cfg = dict(cfg)
        self._c = N.make_config(cfg)
        if isinstance(weights, dict):
            flat = np.concatenate([np.ascontiguousarray(v, dtype=np.float32).ravel()
                                   for v in weights.values()])
        else:
            flat = np.ascontiguousarray(weights, dtype=np.float32).ravel()
        h = C.c_void_p()
        st = N.lib.nv_unet_create(C.byref(self._c), flat.ctypes.data_as(C.c_void_p), flat.size,
                                  C.byref(h))
        N.check(st, "nv_unet_create")
        self._h = h
        self._ws = {}

    def close(self):
        if getattr(self, "_h", None):
            N.lib.nv_unet_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_options(self, graphs=True):
        """nv_unet_set_options: replay denoise steps from captured HIP graphs (default)
        or launch every kernel from the host."""
        N.check(N.lib.nv_unet_set_options(self._h, N.NV_UNET_GRAPHS if graphs else 0),
                "nv_unet_set_options")

    def workspace_bytes(self, B):
        n = int(N.lib.nv_denoise_workspace(self._h, B))
        if n == 0:
            raise N.NvError(N.NV_ERR_INVALID_ARG, "nv_denoise_workspace")
        return n

    def _workspace(self, B, device):
        if B not in self._ws:
            need = self.workspace_bytes(B)
            own, addr = workspace(need, device)
            self._ws[B] = (own, addr, need)
        return self._ws[B]

    def nv_denoise(self, latent, k, cond, uncond, pooled=None, guidance=7.5,
                   sched=(1000, 50, 0.00085, 0.012)):
        """In place: latent [B][C][H][W] f32 holds x_K per sample, returns x_0."""
        _need_cuda(latent, cond, uncond, pooled)
        B = latent.shape[0]
        kk = (C.c_int32 * B)(*[int(v) for v in k])
        s = N.make_schedule(*sched)
        _own, addr, need = self._workspace(B, latent.device)
        st = N.lib.nv_denoise(self._h, C.byref(s), _p(latent), kk, B, _p(cond), _p(uncond),
                              _p(pooled), float(guidance), C.c_void_p(addr), need, _stream())
        N.check(st, "nv_denoise")
        return latent

    def nv_denoise_eta(self, latent, k, cond, uncond, eta, noise, pooled=None, guidance=7.5,
                       sched=(1000, 50, 0.00085, 0.012)):
        """nv_denoise with DDIM's stochastic update: noise f32 [B][N][C][H][W] holds the
        standard normal draws of every sample and grid step."""
        _need_cuda(latent, cond, uncond, pooled, noise)
        B = latent.shape[0]
        if noise.dtype != torch.float32 or tuple(noise.shape[:2]) != (B, sched[1]) or \
                noise[0, 0].numel() != latent[0].numel() or not noise.is_contiguous():
            raise ValueError("noise must be contiguous float32 [B][N][*latent]")
        kk = (C.c_int32 * B)(*[int(v) for v in k])
        s = N.make_schedule(*sched)
        _own, addr, need = self._workspace(B, latent.device)
        st = N.lib.nv_denoise_eta(self._h, C.byref(s), _p(latent), kk, B, _p(cond), _p(uncond),
                                  _p(pooled), float(guidance), float(eta), _p(noise),
                                  C.c_void_p(addr), need, _stream())
        N.check(st, "nv_denoise_eta")
        return latent

    def nv_denoise_store(self, latent, k, cond, uncond, store, slot_k, entry, pooled=None,
                         guidance=7.5, sched=(1000, 50, 0.00085, 0.012)):
        """nv_denoise that also copies each sample's state after slot_k[s] steps to
        store[entry[b]][s] (store: f32 [n_store][n_slots][C][H][W]; entry[b] = -1: none)."""
        _need_cuda(latent, cond, uncond, pooled, store)
        B = latent.shape[0]
        kk = (C.c_int32 * B)(*[int(v) for v in k])
        sk = (C.c_int32 * len(slot_k))(*[int(v) for v in slot_k])
        ee = (C.c_int64 * B)(*[int(v) for v in entry])
        s = N.make_schedule(*sched)
        _own, addr, need = self._workspace(B, latent.device)
        st = N.lib.nv_denoise_store(self._h, C.byref(s), _p(latent), kk, B, _p(cond), _p(uncond),
                                    _p(pooled), float(guidance), _p(store), store.shape[0],
                                    len(slot_k), sk, ee, C.c_void_p(addr), need, _stream())
        N.check(st, "nv_denoise_store")
        return latent

    def nv_denoise_store_pool(self, latent, k, cond, uncond, pool, slot_k, dst, pooled=None,
                              guidance=7.5, sched=(1000, 50, 0.00085, 0.012)):
        """nv_denoise that also copies each sample's state after slot_k[s] steps to
        pool[dst[b][s]] (pool: f32 [n_pool][C][H][W]; dst host [B][n_slots], -1: none)."""
        _need_cuda(latent, cond, uncond, pooled, pool)
        B = latent.shape[0]
        kk = (C.c_int32 * B)(*[int(v) for v in k])
        sk = (C.c_int32 * len(slot_k))(*[int(v) for v in slot_k])
        dd = np.ascontiguousarray(dst, dtype=np.int32).reshape(B, len(slot_k))
        s = N.make_schedule(*sched)
        _own, addr, need = self._workspace(B, latent.device)
        st = N.lib.nv_denoise_store_pool(self._h, C.byref(s), _p(latent), kk, B, _p(cond),
                                         _p(uncond), _p(pooled), float(guidance), _p(pool),
                                         pool.shape[0], len(slot_k), sk, dd.ctypes.data,
                                         C.c_void_p(addr), need, _stream())
        N.check(st, "nv_denoise_store_pool")
        return latent

    def nv_unet_eps(self, x, step_idx, cond, uncond, pooled=None,
                    sched=(1000, 50, 0.00085, 0.012)):
        """Per-row epsilon of one evaluation: (eps_uncond, eps_cond) [B][C][H][W] f32."""
        _need_cuda(x, cond, uncond, pooled)
        B = x.shape[0]
        si = (C.c_int32 * B)(*[int(v) for v in step_idx])
        s = N.make_schedule(*sched)
        eu = torch.empty((B, self.cfg["out_ch"], self.cfg["H"], self.cfg["W"]),
                         dtype=torch.float32, device=x.device)
        ec = torch.empty_like(eu)
        _own, addr, need = self._workspace(B, x.device)
        st = N.lib.nv_unet_eps(self._h, C.byref(s), _p(x), si, B, _p(cond), _p(uncond),
                               _p(pooled), _p(eu), _p(ec), C.c_void_p(addr), need, _stream())
        N.check(st, "nv_unet_eps")
        return eu, ec


_op_ws = {}


def _op_workspace(device):
    key = str(device)
    if key not in _op_ws:
        need = int(N.lib.nv_op_workspace())
        own, addr = workspace(need, device)
        _op_ws[key] = (own, addr, need)
    return _op_ws[key]


def nv_op_linear(x, w, bias=None, residual=None, out=None, x2=None):
    """out[M][N] = [x | x2][M][K] w[N][K]^T (+bias) (+residual); float16, bias float32."""
    _need_cuda(x, w, x2)
    M, K1 = x.shape
    K2 = x2.shape[1] if x2 is not None else 0
    Nn = w.shape[0]
    if out is None:
        out = torch.empty((M, Nn), dtype=torch.float16, device=x.device)
    _own, addr, need = _op_workspace(x.device)
    st = N.lib.nv_op_linear(_p(x), _p(x2), _p(w), _p(bias), _p(residual), _p(out), M, Nn, K1, K2,
                            C.c_void_p(addr), need, _stream())
    N.check(st, "nv_op_linear")
    return out


def nv_op_conv3x3(x, w, bias=None, stride=1, upsample=False, out=None, x2=None):
    """NHWC float16 3x3 conv of [x | x2]: x [B][H][W][Cin1], w [Cout][3][3][Cin] -> [B][Ho][Wo][Cout]."""
    _need_cuda(x, w, x2)
    B, H, W, Cin1 = x.shape
    Cin2 = x2.shape[3] if x2 is not None else 0
    Cout = w.shape[0]
    Ho, Wo = (2 * H, 2 * W) if upsample else (H // stride, W // stride)
    if out is None:
        out = torch.empty((B, Ho, Wo, Cout), dtype=torch.float16, device=x.device)
    _own, addr, need = _op_workspace(x.device)
    st = N.lib.nv_op_conv3x3(_p(x), _p(x2), _p(w), _p(bias), _p(out), B, H, W, Cin1, Cin2, Cout,
                             stride, int(bool(upsample)), C.c_void_p(addr), need, _stream())
    N.check(st, "nv_op_conv3x3")
    return out

def nv_op_attention(q, k, vt, heads, scale, L=None, vt_row=None, out=None):
    """Multi-head attention of q [rows][S][C] over keys k [rows][L][C] and values
    given transposed, vt [C][rows * vt_row] (key j of row r in column r * vt_row + j);
    float16 in and out."""
    _need_cuda(q, k, vt)
    rows, S, C = q.shape
    L = k.shape[1] if L is None else L
    vt_row = vt.shape[1] // rows if vt_row is None else vt_row
    if out is None:
        out = torch.empty((rows, S, C), dtype=torch.float16, device=q.device)
    st = N.lib.nv_op_attention(_p(q), _p(k), _p(vt), _p(out), rows, S, L, heads, C // heads,
                               q.stride(1), k.stride(1), out.stride(1), vt.stride(0), vt_row,
                               float(scale), _stream())
    N.check(st, "nv_op_attention")
    return out


def nv_trace_enable(family_mask, max_launches=65536):
    N.check(N.lib.nv_trace_enable(family_mask, max_launches), "nv_trace_enable")


def nv_trace_disable():
    N.lib.nv_trace_disable()


def nv_trace_records():
    """Every launch of the current trace: list of (family, (m, n, k, variant), ms, flops)."""
    n = C.c_int64()
    ms, fl, by = C.c_double(), C.c_double(), C.c_double()
    N.check(N.lib.nv_trace_read(-1 & 0x7FFFFFFF, C.byref(n), C.byref(ms), C.byref(fl), C.byref(by)),
            "nv_trace_read")
    out = []
    fam = C.c_int32()
    shape = (C.c_int64 * 4)()
    for i in range(n.value):
        N.check(N.lib.nv_trace_get(i, C.byref(fam), shape, C.byref(ms), C.byref(fl)),
                "nv_trace_get")
        out.append((fam.value, tuple(shape), ms.value, fl.value))
    return out


def nv_trace_read(family):
    """(launches, ms, flops, bytes) summed over the recorded launches of `family`."""
    n = C.c_int64()
    ms, fl, by = C.c_double(), C.c_double(), C.c_double()
    N.check(N.lib.nv_trace_read(family, C.byref(n), C.byref(ms), C.byref(fl), C.byref(by)),
            "nv_trace_read")
    return int(n.value), ms.value, fl.value, by.value


def nv_probe_peaks(device=None):
    """Measured dense matrix-core throughput (float16 and bfloat16, TFLOP/s) from
    nv_probe_mfma and HBM read bandwidth (GB/s) from nv_probe_read over 4 GiB;
    each timed after a full-size warm-up launch."""
    dev = torch.device(device or "cuda:0")
    sink = torch.zeros(256, dtype=torch.float32, device=dev)
    ev = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    out = {}
    blocks, iters = 2048, 4096
    for name, bf in (("f16", 0), ("bf16", 1)):
        for timed in (False, True):
            e0, e1 = ev()
            e0.record()
            N.check(N.lib.nv_probe_mfma(bf, iters, blocks, _p(sink), _stream()), "nv_probe_mfma")
            e1.record()
            torch.cuda.synchronize()
        out[name + "_tflops"] = blocks * 4 * iters * 8 * 16384 / (e0.elapsed_time(e1) * 1e-3) / 1e12
    buf = torch.empty(1 << 32, dtype=torch.uint8, device=dev)
    for timed in (False, True):
        e0, e1 = ev()
        e0.record()
        N.check(N.lib.nv_probe_read(_p(buf), buf.numel(), 8192, _p(sink), _stream()),
                "nv_probe_read")
        e1.record()
        torch.cuda.synchronize()
    out["hbm_read_gbps"] = buf.numel() / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del buf
    return out


def nv_cache_insert(rows, cache, n, entry=None, payload=None):
    """Append f32 rows [m][d] to cache (f32, or bf16 bits / torch.bfloat16) at row n, and
    payload[n + i] = entry[i] when both are given (int32 device tensors).  Returns n + m."""
    _need_cuda(rows, cache, entry, payload)
    assert rows.dtype == torch.float32 and rows.is_contiguous() and cache.is_contiguous()
    m, d = rows.shape
    cdt = N.NV_F32 if cache.dtype == torch.float32 else N.NV_BF16
    if cdt == N.NV_BF16 and cache.dtype not in BF16_DTYPES:
        raise ValueError("cache must be float32 or bfloat16 (bits)")
    st = N.lib.nv_cache_insert(_p(rows), m, d, _p(cache), cdt, int(n), cache.shape[0], _p(entry),
                               _p(payload), _stream())
    N.check(st, "nv_cache_insert")
    return int(n) + m
