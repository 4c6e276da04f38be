"""Match predictor: a linear one-class SVM over the cached prompt embeddings
(test infrastructure only).

Follows Sec. 5.2 and Sec. 6: a one-class SVM trained by stochastic gradient
descent on every embedding in the vector DB (all labelled as inliers), with
nu = 0.001; a request goes to the cache lookup only when the classifier says
a close match is likely, else it is generated from scratch (Alg. 1).

Definitions used (readings; the paper names the model, not its equations):
  * the linear one-class SVM in its primal form with slack folded in:
        J(w, rho) = nu/2 |w|^2 - nu rho + (1/n) sum_i max(0, rho - w.x_i);
    its decision value is s(q) = w.q - rho, and the prediction is s(q) >= tau
    (tau = 0 by default; the threshold is the precision / recall knob);
  * plain SGD on J, one sample at a time in a visiting order the caller
    draws, from w = 0, rho = 0, with step eta_t = eta0 / (1 + eta0 nu t);
    the hinge counts as active when rho - w.x > 0;
  * arithmetic in float64; w.x is summed left to right over the d products
    (each product rounded), so the same steps give the same bits anywhere.
"""
import numpy as np


def as_f64(rows):
    rows = np.asarray(rows)
    if rows.dtype == np.uint16:  # bfloat16 bit patterns
        rows = (rows.astype(np.uint32) << 16).view(np.float32)
    return rows.astype(np.float64)


def seq_dot(w, x):
    """w.x: products rounded to float64, summed strictly left to right."""
    return float(np.cumsum(w * x)[-1]) if len(w) else 0.0


def objective(w, rho, X, nu):
    X = as_f64(X)
    margins = rho - X @ w
    return 0.5 * nu * float(w @ w) - nu * rho + float(np.maximum(0.0, margins).mean())


def train(X, nu, order, eta0=1.0):
    """SGD on J over the rows of X (float32 or bfloat16 bits [n][d]) in the given
    visiting order.  Returns (w float64 [d], rho)."""
    X = as_f64(X)
    w = np.zeros(X.shape[1])
    rho = 0.0
    for t, i in enumerate(order):
        x = X[int(i)]
        eta = eta0 / (1.0 + eta0 * nu * t)
        if rho - seq_dot(w, x) > 0.0:
            w = w - eta * (nu * w - x)
            rho = rho - eta * (1.0 - nu)
        else:
            w = w - eta * (nu * w)
            rho = rho + eta * nu
    return w, rho


def scores(w, rho, Q):
    """Decision values s(q) = w.q - rho (float64, left-to-right dot) per query row."""
    Q = as_f64(Q)
    return np.array([seq_dot(w, q) - rho for q in Q])


def predict(w, rho, Q, tau=0.0):
    """True where a close match is predicted (s(q) >= tau)."""
    return scores(w, rho, Q) >= tau
