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
