"""Oracle: per-chunk gradients (test infrastructure only).

Sec. 1 ("Background") defines the chunk gradient g_{D_j} as the sum over the
samples of D_j of the per-sample gradient of the prediction error l, and
grad L = sum_j g_{D_j} (the 1/N~ normalisation dropped, as the paper does when
it introduces g_{D_j}).  The paper leaves l open; the two losses used here are
    linear    l(x, y, w) = (x.w - y)^2 / 2            grad = x (x.w - y)
    logistic  l(x, y, w) = -y log s(x.w) - (1-y) log(1 - s(x.w)),
              s(z) = 1 / (1 + e^-z),                  grad = x (s(x.w) - y)
Everything is computed in fp64 from the stored fp32 inputs.
"""
from __future__ import annotations

import numpy as np


def sigmoid(z: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-z))


def chunk_gradient(Xi: np.ndarray, yi: np.ndarray, w: np.ndarray, loss: str) -> np.ndarray:
    """g_{D_i} = X_i^T r_i with residual r_i = X_i w - y_i (linear) or s(X_i w) - y_i (logistic)."""
    Xi = np.asarray(Xi, dtype=np.float64)
    z = Xi @ np.asarray(w, dtype=np.float64)
    y = np.asarray(yi, dtype=np.float64)
    if loss == "linear":
        r = z - y
    elif loss == "logistic":
        r = sigmoid(z) - y
    else:
        raise ValueError(loss)
    return Xi.T @ r


def chunk_gradients(X: np.ndarray, y: np.ndarray, W: np.ndarray, loss: str) -> np.ndarray:
    """G [N][d] for one evaluation point w, or [b][N][d] for b points W [b][d]."""
    W = np.asarray(W)
    if W.ndim == 1:
        return np.stack([chunk_gradient(X[i], y[i], W, loss) for i in range(X.shape[0])])
    return np.stack([chunk_gradients(X, y, W[q], loss) for q in range(W.shape[0])])

