"""CPU-side checks of the C ABI: the library loads, exports every declared
symbol, enumerates the same parameters as the input generator, and rejects
bad arguments before launching anything (no GPU is touched here)."""
import ctypes as C
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "nv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = set(re.findall(r"\b(nv_[a-z0-9_]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    from paper_2312_04429_amd import _native as N
    names = _declared()
    assert {"nv_cache_lookup", "nv_denoise", "nv_unet_create", "nv_gather_states"} <= names
    for n in names:
        assert hasattr(N.lib, n), n
    assert set(N.EXPORTS) == names
    assert N.lib.nv_version().decode().startswith("nv ")


@pytest.mark.parametrize("name", ["tiny", "sd15", "sdxl"])
def test_param_enumeration_matches_generator(name):
    import paper_2312_04429_amd as P
    cfg = synth.unet_config(name)
    specs = synth.param_specs(cfg)
    assert P.nv_unet_param_count(cfg) == synth.param_count(cfg)
    for i in list(range(0, len(specs), max(1, len(specs) // 97))) + [len(specs) - 1]:
        nm, numel = P.nv_unet_param_info(cfg, i)
        sn, shape, _ = specs[i]
        assert nm == sn
        n = 1
        for s in shape:
            n *= s
        assert numel == n


def test_invalid_configs_rejected():
    import paper_2312_04429_amd as P
    bad = [dict(ch=(30, 64)), dict(H=15), dict(n_heads=3), dict(gn_groups=7), dict(pooled_dim=77),
           dict(n_res=0)]
    for over in bad:
        assert P.nv_unet_param_count(synth.unet_config("tiny", **over)) == -1, over


def test_lookup_validation_before_launch():
    from paper_2312_04429_amd import _native as N
    lib = N.lib
    thr = (C.c_float * 2)(0.9, 0.75)
    kv = (C.c_int32 * 2)(10, 5)
    dummy = C.c_void_p(0x10000)
    args = lambda **o: dict(dict(q=dummy, m=4, cache=dummy, dt=N.NV_BF16, n=100, d=64, thr=thr,
                                 kv=kv, J=2, idx=dummy, sim=dummy, k=dummy, ws=dummy,
                                 wsb=1 << 30), **o)

    def call(a):
        return lib.nv_cache_lookup(a["q"], a["m"], a["cache"], a["dt"], a["n"], a["d"], a["thr"],
                                   a["kv"], a["J"], a["idx"], a["sim"], a["k"], a["ws"], a["wsb"],
                                   None)
    assert call(args(q=None)) == N.NV_ERR_INVALID_ARG
    assert call(args(m=0)) == N.NV_ERR_INVALID_ARG
    assert call(args(n=-1)) == N.NV_ERR_INVALID_ARG
    assert call(args(dt=7)) == N.NV_ERR_INVALID_ARG
    assert call(args(J=0)) == N.NV_ERR_INVALID_ARG
    assert call(args(thr=(C.c_float * 2)(0.75, 0.9))) == N.NV_ERR_INVALID_ARG
    assert call(args(thr=(C.c_float * 2)(float("nan"), 0.1))) == N.NV_ERR_INVALID_ARG
    assert call(args(kv=(C.c_int32 * 2)(10, -1))) == N.NV_ERR_INVALID_ARG
    assert call(args(d=60)) == N.NV_ERR_UNSUPPORTED
    assert call(args(d=4096)) == N.NV_ERR_UNSUPPORTED
    assert call(args(ws=None)) == N.NV_ERR_WORKSPACE
    assert call(args(wsb=16)) == N.NV_ERR_WORKSPACE
    assert call(args(ws=C.c_void_p(0x10010))) == N.NV_ERR_WORKSPACE
    assert "workspace" in lib.nv_last_error().decode()
    assert lib.nv_cache_lookup_workspace(8, 1_000_000, 768) > 0
    assert lib.nv_status_string(-5).decode().startswith("workspace")


def test_unet_entry_points_reject_null_handles():
    from paper_2312_04429_amd import _native as N
    s = N.make_schedule(1000, 50, 0.00085, 0.012)
    k = (C.c_int32 * 1)(5)
    d = C.c_void_p(0x10000)
    assert N.lib.nv_denoise(None, C.byref(s), d, k, 1, d, d, None, 7.5, d, 1 << 30, None) == \
        N.NV_ERR_INVALID_ARG
    assert N.lib.nv_denoise_workspace(None, 1) == 0
    assert N.lib.nv_gather_states(d, 10, 0, None, None, 10, d, d, d, 1, 16, d, None) == \
        N.NV_ERR_INVALID_ARG
    cfg = N.make_config(synth.unet_config("tiny", ch=(30, 64)))
    h = C.c_void_p()
    assert N.lib.nv_unet_create(C.byref(cfg), d, 10, C.byref(h)) == N.NV_ERR_INVALID_ARG


def test_pool_entry_points_validate_before_launch():
    """Hole-aware fetch, table updates, row moves and the pool-storing denoise reject
    bad arguments synchronously (no GPU touched); empty updates / moves are no-ops."""
    from paper_2312_04429_amd import _native as N
    lib = N.lib
    d = C.c_void_p(0x10000)
    sk = (C.c_int32 * 2)(5, 10)

    def gp(**o):
        a = dict(pool=d, n_pool=4, table=d, n_ent=4, S=2, sk=sk, payload=d, n_rows=4, idx=d,
                 k=d, noise=d, B=1, lat=16, out=d)
        a.update(o)
        return lib.nv_gather_pool(a["pool"], a["n_pool"], a["table"], a["n_ent"], a["S"],
                                  a["sk"], a["payload"], a["n_rows"], a["idx"], a["k"],
                                  a["noise"], a["B"], a["lat"], a["out"], None)
    assert gp(idx=None) == N.NV_ERR_INVALID_ARG
    assert gp(B=0) == N.NV_ERR_INVALID_ARG
    assert gp(lat=18) == N.NV_ERR_INVALID_ARG
    assert gp(pool=None) == N.NV_ERR_INVALID_ARG
    assert gp(table=None) == N.NV_ERR_INVALID_ARG
    assert gp(S=0) == N.NV_ERR_INVALID_ARG
    assert gp(sk=(C.c_int32 * 2)(5, 0)) == N.NV_ERR_INVALID_ARG
    assert gp(payload=None, n_rows=5) == N.NV_ERR_INVALID_ARG
    assert gp(out=C.c_void_p(0x10004)) == N.NV_ERR_INVALID_ARG
    assert lib.nv_table_update(None, 4, 2, None, 0, None) == N.NV_OK
    assert lib.nv_table_update(None, 4, 2, d, 1, None) == N.NV_ERR_INVALID_ARG
    assert lib.nv_table_update(d, 4, 17, d, 1, None) == N.NV_ERR_INVALID_ARG
    assert lib.nv_cache_move_rows(None, N.NV_BF16, 4, 8, None, None, None, 0, None) == N.NV_OK
    assert lib.nv_cache_move_rows(d, N.NV_BF16, 4, 7, None, d, d, 1, None) == N.NV_ERR_INVALID_ARG
    assert lib.nv_cache_move_rows(d, 3, 4, 8, None, d, d, 1, None) == N.NV_ERR_INVALID_ARG
    assert lib.nv_cache_move_rows(d, N.NV_F32, 4, 8, None, None, d, 1, None) == \
        N.NV_ERR_INVALID_ARG
    s = N.make_schedule(1000, 50, 0.00085, 0.012)
    k = (C.c_int32 * 1)(0)
    dst = (C.c_int32 * 2)(0, 1)
    assert lib.nv_denoise_store_pool(None, C.byref(s), d, k, 1, d, d, None, 7.5, d, 2, 2, sk,
                                     None, d, 1 << 30, None) == N.NV_ERR_INVALID_ARG
    assert lib.nv_denoise_store_pool(None, C.byref(s), d, k, 65, d, d, None, 7.5, d, 2, 2, sk,
                                     dst, d, 1 << 30, None) == N.NV_ERR_INVALID_ARG


def test_static_lookup_validation_before_launch():
    """nv_cache_lookup_static rejects bad arguments, and lookups needing more
    scratch than its 64 MiB array, before touching a device."""
    from paper_2312_04429_amd import _native as N
    lib = N.lib
    thr = (C.c_float * 2)(0.9, 0.75)
    kv = (C.c_int32 * 2)(10, 5)
    dummy = C.c_void_p(0x10000)

    def call(q=dummy, m=4, n=100, d=64, dt=N.NV_BF16, J=2):
        return lib.nv_cache_lookup_static(q, m, dummy, dt, n, d, thr, kv, J, dummy, dummy, dummy,
                                          None)
    assert call(q=None) == N.NV_ERR_INVALID_ARG
    assert call(m=0) == N.NV_ERR_INVALID_ARG
    assert call(J=0) == N.NV_ERR_INVALID_ARG
    assert call(d=60) == N.NV_ERR_UNSUPPORTED
    # 256 queries over 5M rows of 768 bf16 dims need about 80 MiB of scratch
    assert lib.nv_cache_lookup_workspace(256, 5_000_000, 768) > N.NV_LOOKUP_STATIC_BYTES
    assert call(m=256, n=5_000_000, d=768) == N.NV_ERR_UNSUPPORTED
    # the limits quoted with the declaration
    assert lib.nv_cache_lookup_workspace(8, 85_000_000, 768) <= N.NV_LOOKUP_STATIC_BYTES
    assert lib.nv_cache_lookup_workspace(256, 4_100_000, 768) <= N.NV_LOOKUP_STATIC_BYTES


def test_gated_lookup_validation_before_launch():
    """nv_cache_lookup_gated checks the lookup's arguments, the predictor's and
    the workspace before any launch."""
    from paper_2312_04429_amd import _native as N
    lib = N.lib
    thr = (C.c_float * 2)(0.9, 0.75)
    kv = (C.c_int32 * 2)(10, 5)
    dummy = C.c_void_p(0x10000)
    searched = C.c_int32(-7)
    need = lib.nv_cache_lookup_gated_workspace(4, 100, 64)
    assert need >= lib.nv_cache_lookup_workspace(4, 100, 64) + 4 * 64 * 4

    def call(q=dummy, m=4, d=64, w=dummy, rho=0.5, tau=0.0, ns=C.byref(searched), ws=dummy,
             wb=need):
        return lib.nv_cache_lookup_gated(q, m, dummy, N.NV_BF16, 100, d, thr, kv, 2, w, rho, tau,
                                         dummy, dummy, dummy, None, ns, ws, wb, None)
    assert call(q=None) == N.NV_ERR_INVALID_ARG
    assert call(m=4097) == N.NV_ERR_INVALID_ARG
    assert call(w=None) == N.NV_ERR_INVALID_ARG
    assert call(ns=None) == N.NV_ERR_INVALID_ARG
    assert call(rho=float("inf")) == N.NV_ERR_INVALID_ARG
    assert call(tau=float("nan")) == N.NV_ERR_INVALID_ARG
    assert call(d=60) == N.NV_ERR_UNSUPPORTED
    assert call(wb=need - 1) == N.NV_ERR_WORKSPACE
    assert call(ws=C.c_void_p(0x10008)) == N.NV_ERR_WORKSPACE
    assert searched.value == -7  # untouched on every error
    assert lib.nv_cache_lookup_gated_workspace(0, 100, 64) == 0
