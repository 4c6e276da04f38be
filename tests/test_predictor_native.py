"""The native match-predictor trainer (host C++ behind the C ABI; no GPU)
against the oracle's SGD (Sec. 5.2): identical float64 weights and offset, bit
for bit, on float32 and bfloat16 rows; argument checks of the trainer and the
gate (before any launch)."""
import ctypes as C

import numpy as np
import pytest

import synth
from oracle import predictor as PR


@pytest.mark.parametrize("dtype,nu,n,d,T", [("f32", 0.001, 500, 768, 3000),
                                            ("bf16", 0.001, 300, 768, 2000),
                                            ("f32", 0.3, 40, 3, 5000),
                                            ("bf16", 1.0, 64, 64, 700)])
def test_native_trainer_matches_oracle(dtype, nu, n, d, T):
    import paper_2312_04429_amd as P
    rng = np.random.default_rng(n + d)
    X = synth.make_cache(n, d, 8, 0.1, n, "f32" if dtype == "f32" else "bf16")
    order = rng.integers(0, n, T)
    w, rho = P.nv_ocsvm_train(X, nu, order)
    wo, ro = PR.train(X, nu, order)
    assert np.array_equal(w, wo) and rho == ro


def test_argument_checks():
    import paper_2312_04429_amd as P
    from paper_2312_04429_amd import _native as N
    X = np.ones((4, 8), np.float32)
    for nu in (0.0, -0.1, 1.5):
        with pytest.raises(N.NvError):
            P.nv_ocsvm_train(X, nu, [0, 1])
    with pytest.raises(N.NvError):
        P.nv_ocsvm_train(X, 0.1, [0, 4])
    w, rho = P.nv_ocsvm_train(X, 0.1, [])
    assert not w.any() and rho == 0.0
    d = C.c_void_p(0x10000)
    lib = N.lib
    assert lib.nv_match_gate(None, 1, 8, d, 0.0, 0.0, d, None, None, None, None) == \
        N.NV_ERR_INVALID_ARG
    assert lib.nv_match_gate(d, 0, 8, d, 0.0, 0.0, d, None, None, None, None) == \
        N.NV_ERR_INVALID_ARG
    assert lib.nv_match_gate(d, 1, 8, d, 0.0, 0.0, None, None, None, None, None) == \
        N.NV_ERR_INVALID_ARG
    assert lib.nv_match_gate(d, 1, 8, d, 0.0, 0.0, None, d, None, d, None) == \
        N.NV_ERR_INVALID_ARG
    assert lib.nv_match_gate(d, 1, 8, d, float("inf"), 0.0, d, None, None, None, None) == \
        N.NV_ERR_INVALID_ARG
