"""Pins of the oracle's match predictor (Sec. 5.2, Sec. 6: linear one-class SVM
trained by SGD on the vector DB's embeddings).

Checked against things other than itself: a literal Python loop for the
left-to-right dot; the closed-form optimum when every training point is one
unit vector (w = x, rho = 1); the optimum of the same objective solved as a
constrained QP by scipy (SLSQP on the slack form); the nu-property of the
one-class SVM optimum (at most a nu fraction of training points outside, at
least nu on or outside the boundary); and scikit-learn's SGDOneClassSVM,
the classifier the paper names, on clustered data.
"""
import numpy as np
import pytest
from scipy.optimize import minimize

from oracle import predictor as PR


def test_seq_dot_is_left_to_right():
    rng = np.random.default_rng(0)
    for d in (1, 7, 768):
        w = rng.standard_normal(d)
        x = rng.standard_normal(d).astype(np.float32).astype(np.float64)
        s = 0.0
        for k in range(d):
            s = s + w[k] * x[k]
        assert PR.seq_dot(w, x) == s


def test_single_point_closed_form():
    """All points equal to a unit x: J is minimised at w = x, rho = |x|^2 = 1."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal(8)
    x /= np.linalg.norm(x)
    X = np.tile(x.astype(np.float32), (50, 1))
    w, rho = PR.train(X, 0.5, np.arange(20000) % 50)
    assert np.linalg.norm(w - X[0]) < 0.02 and abs(rho - 1.0) < 0.02
    assert PR.objective(w, rho, X, 0.5) >= -0.25 - 1e-12   # J* = -nu/2


def _qp(X, nu):
    n, d = X.shape
    Xd = X.astype(np.float64)
    f = lambda v: 0.5 * nu * v[:d] @ v[:d] - nu * v[d] + v[d + 1:].mean()
    cons = [{"type": "ineq", "fun": lambda v: v[d + 1:] - (v[d] - Xd @ v[:d])},
            {"type": "ineq", "fun": lambda v: v[d + 1:]}]
    r = minimize(f, np.zeros(d + 1 + n), constraints=cons, method="SLSQP",
                 options={"maxiter": 500, "ftol": 1e-12})
    assert r.success
    return r.x[:d], r.x[d], r.fun


def test_sgd_reaches_the_qp_optimum_and_nu_property():
    rng = np.random.default_rng(0)
    rng.standard_normal(8)
    nu, n, d = 0.2, 40, 3
    X = rng.standard_normal((n, d)).astype(np.float32) + np.array([2, 0, 0], np.float32)
    wq, rq, jq = _qp(X, nu)
    sq = PR.scores(wq, rq, X)
    assert (sq < -1e-7).mean() <= nu <= (sq <= 1e-7).mean()      # nu-property at the optimum
    w, rho = PR.train(X, nu, np.random.default_rng(1).integers(0, n, 100000))
    j = PR.objective(w, rho, X, nu)
    assert jq - 1e-9 <= j <= jq + 1e-3
    assert (PR.scores(w, rho, X) < 0).mean() <= nu


def test_agrees_with_scikit_learn():
    from sklearn.linear_model import SGDOneClassSVM
    rng = np.random.default_rng(2)
    n, d, nu = 2000, 16, 0.1
    centre = np.r_[3.0, np.zeros(d - 1)]
    X = (rng.standard_normal((n, d)) * 0.3 + centre).astype(np.float32)
    sk = SGDOneClassSVM(nu=nu, random_state=0, max_iter=200, tol=None).fit(X)
    w, rho = PR.train(X, nu, np.random.default_rng(3).integers(0, n, 200000))
    T = (rng.standard_normal((4000, d)) * 0.5 + centre).astype(np.float32)
    agree = ((sk.decision_function(T) >= 0) == PR.predict(w, rho, T)).mean()
    assert agree >= 0.99
    out_sk = (sk.decision_function(X) < 0).mean()
    out = (PR.scores(w, rho, X) < 0).mean()
    assert abs(out - out_sk) <= 0.01 and out <= nu


def test_threshold_knob_and_bf16_rows():
    rng = np.random.default_rng(4)
    X = rng.standard_normal((30, 8)).astype(np.float32)
    w, rho = PR.train(X, 0.3, np.arange(300) % 30)
    s = PR.scores(w, rho, X)
    for tau in (-1.0, 0.0, float(np.median(s)), float(s[3])):   # s[3] itself predicts a match
        assert (PR.predict(w, rho, X, tau) == (s >= tau)).all()
    bits = (X.view(np.uint32) >> 16).astype(np.uint16)      # truncation: exact bf16 values
    Xb = (bits.astype(np.uint32) << 16).view(np.float32)
    wa, ra = PR.train(bits, 0.3, np.arange(300) % 30)
    wb, rb = PR.train(Xb, 0.3, np.arange(300) % 30)
    assert np.array_equal(wa, wb) and ra == rb


def test_first_two_steps_by_hand():
    """From w = 0, rho = 0 the margin is exactly 0, which is not an active hinge: the
    first step only raises rho by eta0 nu; the second (eta = eta0 / (1 + eta0 nu)) sees
    margin rho > 0 and pulls w toward x."""
    x = np.array([[0.5, -0.25, 1.0]], np.float32)
    nu = 0.25
    w, rho = PR.train(x, nu, [0])
    assert not w.any() and rho == 0.25
    w, rho = PR.train(x, nu, [0, 0])
    eta = 1.0 / 1.25
    assert np.array_equal(w, eta * x[0].astype(np.float64))
    assert rho == 0.25 - eta * 0.75
