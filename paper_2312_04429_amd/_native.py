"""ctypes binding of libnv.so (the C ABI in include/nv.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch supplies device memory and the current HIP stream.  If the
library has not been built, importing this module raises.
"""
import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("NV_LIB_PATH") or os.path.join(HERE, "libnv.so")

NV_OK, NV_ERR_INVALID_ARG, NV_ERR_UNSUPPORTED = 0, -1, -2
NV_ERR_OUT_OF_MEMORY, NV_ERR_HIP, NV_ERR_WORKSPACE = -3, -4, -5
NV_F32, NV_BF16 = 0, 1
NV_LOOKUP_STATIC_BYTES = 64 << 20
NV_FAM_CONV, NV_FAM_LINEAR, NV_FAM_ATTN, NV_FAM_SCAN = 1, 2, 4, 8
NV_UNET_GRAPHS = 1

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2312_04429_amd.build`")
lib = C.CDLL(LIB_PATH)


class nv_unet_config(C.Structure):
    _fields_ = [("in_ch", C.c_int32), ("out_ch", C.c_int32), ("H", C.c_int32), ("W", C.c_int32),
                ("n_levels", C.c_int32), ("ch", C.c_int32 * 4), ("depth", C.c_int32 * 4),
                ("mid_depth", C.c_int32), ("n_res", C.c_int32), ("n_heads", C.c_int32),
                ("head_dim", C.c_int32), ("gn_groups", C.c_int32), ("ctx_len", C.c_int32),
                ("ctx_dim", C.c_int32), ("pooled_dim", C.c_int32), ("gn_eps", C.c_float),
                ("ln_eps", C.c_float)]


class nv_schedule(C.Structure):
    _fields_ = [("T", C.c_int32), ("N", C.c_int32), ("beta_start", C.c_float),
                ("beta_end", C.c_float)]


VP, I32, I64, SZ, F32 = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t, C.c_float
_sigs = {
    "nv_status_string": (C.c_char_p, [I32]),
    "nv_last_error": (C.c_char_p, []),
    "nv_version": (C.c_char_p, []),
    "nv_cache_lookup_workspace": (SZ, [I32, I64, I32]),
    "nv_cache_lookup": (I32, [VP, I32, VP, I32, I64, I32, VP, VP, I32, VP, VP, VP, VP, SZ, VP]),
    "nv_cache_lookup_static": (I32, [VP, I32, VP, I32, I64, I32, VP, VP, I32, VP, VP, VP, VP]),
    "nv_gather_states": (I32, [VP, I64, I32, VP, VP, I64, VP, VP, VP, I32, I64, VP, VP]),
    "nv_unet_param_count": (I64, [C.POINTER(nv_unet_config)]),
    "nv_unet_param_info": (I32, [C.POINTER(nv_unet_config), I64, C.c_char_p, I32,
                                 C.POINTER(I64)]),
    "nv_unet_create": (I32, [C.POINTER(nv_unet_config), VP, I64, C.POINTER(VP)]),
    "nv_unet_destroy": (None, [VP]),
    "nv_denoise_workspace": (SZ, [VP, I32]),
    "nv_denoise": (I32, [VP, C.POINTER(nv_schedule), VP, VP, I32, VP, VP, VP, F32, VP, SZ, VP]),
    "nv_denoise_store": (I32, [VP, C.POINTER(nv_schedule), VP, VP, I32, VP, VP, VP, F32, VP, I64,
                               I32, VP, VP, VP, SZ, VP]),
    "nv_cache_insert": (I32, [VP, I32, I32, VP, I32, I64, I64, VP, VP, VP]),
    "nv_denoise_eta": (I32, [VP, C.POINTER(nv_schedule), VP, VP, I32, VP, VP, VP, F32, F32, VP,
                             VP, SZ, VP]),
    "nv_denoise_store_pool": (I32, [VP, C.POINTER(nv_schedule), VP, VP, I32, VP, VP, VP, F32,
                                    VP, I64, I32, VP, VP, VP, SZ, VP]),
    "nv_gather_pool": (I32, [VP, I64, VP, I64, I32, VP, VP, I64, VP, VP, VP, I32, I64, VP, VP]),
    "nv_table_update": (I32, [VP, I64, I32, VP, I32, VP]),
    "nv_cache_move_rows": (I32, [VP, I32, I64, I32, VP, VP, VP, I32, VP]),
    "nv_ivf_build_workspace": (SZ, [I64, I32, I32]),
    "nv_ivf_build": (I32, [VP, I32, I64, I32, VP, I32, I32, VP, VP, VP, VP, VP, VP, VP, SZ, VP]),
    "nv_ivf_search_workspace": (SZ, [I32, I32, I32, I64]),
    "nv_ivf_search": (I32, [VP, I32, I32, VP, I32, VP, I32, VP, VP, I64, I32, VP, VP, I32, VP,
                            VP, VP, VP, VP, SZ, VP]),
    "nv_cache_lookup_gated_workspace": (SZ, [I32, I64, I32]),
    "nv_cache_lookup_gated": (I32, [VP, I32, VP, I32, I64, I32, VP, VP, I32, VP, C.c_double,
                                    C.c_double, VP, VP, VP, VP, VP, VP, SZ, VP]),
    "nv_ocsvm_train": (I32, [VP, I32, I64, I32, C.c_double, C.c_double, VP, I64, VP, VP]),
    "nv_match_gate": (I32, [VP, I32, I32, VP, C.c_double, C.c_double, VP, VP, VP, VP, VP]),
    "nv_lcbfu_create": (I32, [I32, VP, I64, I64, C.POINTER(VP)]),
    "nv_lcbfu_destroy": (None, [VP]),
    "nv_lcbfu_access": (I32, [VP, I32, VP, VP]),
    "nv_lcbfu_insert": (I32, [VP, I32, VP, VP, VP, VP, VP, VP, VP, VP]),
    "nv_lcbfu_info": (I32, [VP, VP]),
    "nv_lcbfu_export": (I32, [VP, VP, VP, VP]),
    "nv_unet_set_options": (I32, [VP, I32]),
    "nv_unet_eps": (I32, [VP, C.POINTER(nv_schedule), VP, VP, I32, VP, VP, VP, VP, VP, VP, SZ,
                          VP]),
    "nv_trace_enable": (I32, [I32, I32]),
    "nv_trace_disable": (I32, []),
    "nv_trace_get": (I32, [I32, VP, VP, VP, VP]),
    "nv_trace_read": (I32, [I32, C.POINTER(I64), C.POINTER(C.c_double), C.POINTER(C.c_double),
                            C.POINTER(C.c_double)]),
    "nv_probe_mfma": (I32, [I32, I32, I32, VP, VP]),
    "nv_probe_read": (I32, [VP, I64, I32, VP, VP]),
    "nv_op_workspace": (SZ, []),
    "nv_op_linear": (I32, [VP, VP, VP, VP, VP, VP, I64, I32, I32, I32, VP, SZ, VP]),
    "nv_op_conv3x3": (I32, [VP, VP, VP, VP, VP, I32, I32, I32, I32, I32, I32, I32, I32, VP, SZ,
                            VP]),
    "nv_op_attention": (I32, [VP, VP, VP, VP, I32, I32, I32, I32, I32, I32, I32, I32, I64, I64,
                              F32, VP]),
}
for _name, (_res, _args) in _sigs.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTS = tuple(_sigs)


class NvError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = lib.nv_status_string(status).decode()
        detail = lib.nv_last_error().decode()
        super().__init__(f"{where}: {msg} ({status}): {detail}")


def check(status, where):
    if status != NV_OK:
        raise NvError(status, where)


def make_config(cfg):
    c = nv_unet_config()
    c.in_ch, c.out_ch, c.H, c.W = cfg["in_ch"], cfg["out_ch"], cfg["H"], cfg["W"]
    L = len(cfg["ch"])
    c.n_levels = L
    for i in range(4):
        c.ch[i] = cfg["ch"][i] if i < L else 0
        c.depth[i] = cfg["depth"][i] if i < L else 0
    c.mid_depth, c.n_res = cfg["mid_depth"], cfg["n_res"]
    c.n_heads, c.head_dim, c.gn_groups = cfg["n_heads"], cfg["head_dim"], cfg["gn_groups"]
    c.ctx_len, c.ctx_dim, c.pooled_dim = cfg["ctx_len"], cfg["ctx_dim"], cfg["pooled_dim"]
    c.gn_eps, c.ln_eps = cfg["gn_eps"], cfg["ln_eps"]
    return c


def make_schedule(T, N, beta_start, beta_end):
    s = nv_schedule()
    s.T, s.N, s.beta_start, s.beta_end = T, N, beta_start, beta_end
    return s
