"""Worker minibatch gradients, float64 (Sect. 2, Eq. gradient).

Worker i holds minibatch X_i [B][d] with labels y_i [B] and computes, at the
common parameter vector w_t,

    g_i = (1/B) * sum_{x in minibatch} grad f(x, w_t)
    loss_i = (1/B) * sum_{x in minibatch} f(x, w_t)

with f the natural-log cross-entropy of a softmax.  The per-worker loss is
what a worker reports to the PS for the loss estimate F_hat (Sect. 3.1).

Parameter layouts (readings of an unspecified layout):
* softmax regression: W [d][C] row-major, no bias; P = d*C.
* MLP d-H-C with ReLU: flat [W1 (d x H) | b1 (H) | W2 (H x C) | b2 (C)];
  the ReLU derivative at 0 is taken as 0.

Test infrastructure only (see the package docstring).
"""
from __future__ import annotations

import numpy as np


def _softmax_ce(Z: np.ndarray, y: np.ndarray):
    """Row softmax with max subtraction.  Returns (P, per-row CE loss)."""
    zmax = Z.max(axis=1, keepdims=True)
    E = np.exp(Z - zmax)
    s = E.sum(axis=1, keepdims=True)
    P = E / s
    rows = np.arange(Z.shape[0])
    ce = (zmax[:, 0] + np.log(s[:, 0])) - Z[rows, y]
    return P, ce


def _onehot(y: np.ndarray, C: int) -> np.ndarray:
    Y = np.zeros((y.shape[0], C))
    Y[np.arange(y.shape[0]), y] = 1.0
    return Y


def softmax_worker_grads(w: np.ndarray, Xt: np.ndarray, yt: np.ndarray, C: int):
    """Softmax regression.  w [d*C]; Xt [n][B][d]; yt [n][B] in [0, C).

    Returns G float64 [n][d*C] (row i = g_i laid out like W) and loss [n].
    """
    n, B, d = Xt.shape
    W = np.asarray(w, dtype=np.float64).reshape(d, C)
    G = np.empty((n, d * C))
    loss = np.empty(n)
    for i in range(n):
        X = np.asarray(Xt[i], dtype=np.float64)
        y = np.asarray(yt[i], dtype=np.int64)
        P, ce = _softmax_ce(X @ W, y)
        R = (P - _onehot(y, C)) / B          # d(mean CE)/dZ
        G[i] = (X.T @ R).ravel()
        loss[i] = ce.mean()
    return G, loss


def mlp_split(w: np.ndarray, d: int, H: int, C: int):
    w = np.asarray(w, dtype=np.float64)
    o = 0
    W1 = w[o:o + d * H].reshape(d, H); o += d * H
    b1 = w[o:o + H]; o += H
    W2 = w[o:o + H * C].reshape(H, C); o += H * C
    b2 = w[o:o + C]; o += C
    assert o == w.size, "parameter vector length does not match d, H, C"
    return W1, b1, W2, b2


def mlp_worker_grads(w: np.ndarray, Xt: np.ndarray, yt: np.ndarray, H: int, C: int,
                     return_preact: bool = False):
    """Two-layer ReLU MLP.  Returns G [n][P] (flattened like w), loss [n] and,
    on request, the hidden pre-activations A [n][B][H] (the ReLU decisions)."""
    n, B, d = Xt.shape
    W1, b1, W2, b2 = mlp_split(w, d, H, C)
    P_ = w.size
    G = np.empty((n, P_))
    loss = np.empty(n)
    A_all = np.empty((n, B, H)) if return_preact else None
    for i in range(n):
        X = np.asarray(Xt[i], dtype=np.float64)
        y = np.asarray(yt[i], dtype=np.int64)
        A = X @ W1 + b1
        on = A > 0.0
        Hh = np.where(on, A, 0.0)
        P, ce = _softmax_ce(Hh @ W2 + b2, y)
        R = (P - _onehot(y, C)) / B
        dW2 = Hh.T @ R
        db2 = R.sum(axis=0)
        dA = (R @ W2.T) * on
        dW1 = X.T @ dA
        db1 = dA.sum(axis=0)
        G[i] = np.concatenate([dW1.ravel(), db1, dW2.ravel(), db2])
        loss[i] = ce.mean()
        if return_preact:
            A_all[i] = A
    if return_preact:
        return G, loss, A_all
    return G, loss


def worker_grads(cfg, w, Xt, yt):
    """Dispatch on the workload's model."""
    if cfg.model == "softmax":
        return softmax_worker_grads(w, Xt, yt, cfg.C)
    return mlp_worker_grads(w, Xt, yt, cfg.H, cfg.C)
