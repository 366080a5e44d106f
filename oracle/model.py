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
* CNN for 28 x 28 single-channel images (Sect. 4: two convolutional layers
  with 5 x 5 filters and two fully connected layers; the widths are a
  reading): conv 1 -> 20 channels, 2 x 2 max pooling, ReLU, conv 20 -> 50,
  2 x 2 max pooling, ReLU, flatten (channel, row, column) to 800, FC
  800 -> H with ReLU, FC H -> C.  Convolutions are "valid" with stride 1:
  out[o][y][x] = b[o] + sum_{c,u,v} in[c][y+u][x+v] W[o][c][u][v].  A pooling
  window passes its largest value; among equal values the first in
  row-major order of the window, which also receives the gradient.  Flat
  [Wf1 (800 x H) | bf1 | Wf2 (H x C) | bf2 | Wc1 (20x1x5x5) | bc1 |
  Wc2 (50x20x5x5) | bc2]: the fully connected part first, laid out like
  the MLP.

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
                     return_preact: bool = False, decisions: dict | None = None):
    """Two-layer ReLU MLP.  Returns G [n][P] (flattened like w), loss [n] and,
    on request, the hidden pre-activations A [n][B][H] (the ReLU decisions).

    decisions (n = 1 only): {"on": [B][H] booleans} replaces the ReLU
    decisions [A > 0], for tests that accept either outcome of a decision
    taken within rounding; the network is then the same composition with
    those units fixed on or off."""
    n, B, d = Xt.shape
    assert not decisions or n == 1
    W1, b1, W2, b2 = mlp_split(w, d, H, C)
    P_ = w.size
    G = np.empty((n, P_))
    loss = np.empty(n)
    A_all = np.empty((n, B, H)) if return_preact else None
    for i in range(n):
        X = np.asarray(Xt[i], dtype=np.float64)
        y = np.asarray(yt[i], dtype=np.int64)
        A = X @ W1 + b1
        on = decisions["on"] if decisions else A > 0.0
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


CNN_IMG, CNN_K, CNN_C1, CNN_C2 = 28, 5, 20, 50
CNN_FEAT = CNN_C2 * 4 * 4            # after the second pooling: 50 x 4 x 4


def cnn_param_count(H: int, C: int) -> int:
    return (CNN_C1 * CNN_K * CNN_K + CNN_C1 + CNN_C2 * CNN_C1 * CNN_K * CNN_K + CNN_C2
            + CNN_FEAT * H + H + H * C + C)


def cnn_split(w: np.ndarray, H: int, C: int):
    w = np.asarray(w, dtype=np.float64)
    k = CNN_K
    shapes = [(CNN_FEAT, H), (H,), (H, C), (C,),
              (CNN_C1, 1, k, k), (CNN_C1,), (CNN_C2, CNN_C1, k, k), (CNN_C2,)]
    out, o = [], 0
    for sh in shapes:
        m = int(np.prod(sh))
        out.append(w[o:o + m].reshape(sh))
        o += m
    assert o == w.size, "parameter vector length does not match the CNN"
    Wf1, bf1, Wf2, bf2, Wc1, bc1, Wc2, bc2 = out
    return Wc1, bc1, Wc2, bc2, Wf1, bf1, Wf2, bf2


def im2col(X: np.ndarray, k: int) -> np.ndarray:
    """The k x k patches of X [B][Ci][h][w] as a matrix with one row per output
    position (b, y, x) and one column per (c, u, v): X[b][c][y+u][x+v]."""
    B, Ci, h, wd = X.shape
    ho, wo = h - k + 1, wd - k + 1
    win = np.lib.stride_tricks.sliding_window_view(X, (k, k), axis=(2, 3))   # [B][Ci][ho][wo][k][k]
    return win.transpose(0, 2, 3, 1, 4, 5).reshape(B * ho * wo, Ci * k * k)


def conv_valid(X: np.ndarray, W: np.ndarray, b: np.ndarray):
    """X [B][Ci][h][w], W [Co][Ci][k][k] -> out [B][Co][h-k+1][w-k+1] (the
    definition above, as patches times filters) and the patch matrix."""
    B, Ci, h, wd = X.shape
    Co, _, k, _ = W.shape
    ho, wo = h - k + 1, wd - k + 1
    cols = im2col(X, k)
    out = (cols @ W.reshape(Co, -1).T).reshape(B, ho, wo, Co).transpose(0, 3, 1, 2)
    return out + b[None, :, None, None], cols


def conv_weight_grad(dOut: np.ndarray, cols: np.ndarray, W_shape):
    """dW[o][c][u][v] = sum over (b, y, x) of dOut[b][o][y][x] X[b][c][y+u][x+v]."""
    Co = dOut.shape[1]
    dmat = dOut.transpose(0, 2, 3, 1).reshape(-1, Co)
    return (dmat.T @ cols).reshape(W_shape)


def conv_input_grad(dOut: np.ndarray, W: np.ndarray, h: int, wd: int):
    """Gradient of conv_valid with respect to its input: dX[b][c][y+u][x+v] +=
    dOut[b][o][y][x] W[o][c][u][v]."""
    B, Co, ho, wo = dOut.shape
    _, Ci, k, _ = W.shape
    dcols = (dOut.transpose(0, 2, 3, 1).reshape(-1, Co) @ W.reshape(Co, -1)).reshape(B, ho, wo, Ci, k, k)
    dX = np.zeros((B, Ci, h, wd))
    for u in range(k):
        for v in range(k):
            dX[:, :, u:u + ho, v:v + wo] += dcols[:, :, :, :, u, v].transpose(0, 3, 1, 2)
    return dX


def maxpool2(Z: np.ndarray):
    """2 x 2 max pooling, stride 2.  Returns the pooled values and the code
    0..3 of the passing entry ((0,0), (0,1), (1,0), (1,1) in that order;
    the first of equal values)."""
    win = np.stack([Z[:, :, 0::2, 0::2], Z[:, :, 0::2, 1::2], Z[:, :, 1::2, 0::2], Z[:, :, 1::2, 1::2]])
    code = np.argmax(win, axis=0)                                   # first occurrence
    return np.take_along_axis(win, code[None], axis=0)[0], code


def pool_take(Z: np.ndarray, code: np.ndarray):
    """The entries of each 2 x 2 window that the codes name."""
    win = np.stack([Z[:, :, 0::2, 0::2], Z[:, :, 0::2, 1::2], Z[:, :, 1::2, 0::2], Z[:, :, 1::2, 1::2]])
    return np.take_along_axis(win, code[None], axis=0)[0]


def maxpool2_grad(dP: np.ndarray, code: np.ndarray):
    """The pooled gradient placed at each window's passing entry."""
    B, Ch, h, wd = dP.shape
    dZ = np.zeros((B, Ch, 2 * h, 2 * wd))
    for c, (dy, dx) in enumerate(((0, 0), (0, 1), (1, 0), (1, 1))):
        dZ[:, :, dy::2, dx::2] = np.where(code == c, dP, 0.0)
    return dZ


def cnn_worker_grads(w: np.ndarray, Xt: np.ndarray, yt: np.ndarray, H: int, C: int,
                     return_preact: bool = False, decisions: dict | None = None):
    """The CNN above.  Xt [n][B][784] (row-major 28 x 28 images).  Returns
    G [n][P] flattened like w, loss [n] and, on request, per worker the
    values its decisions were taken on: {"Z1": conv1 outputs [B][20][24][24],
    "Z2": conv2 outputs [B][50][8][8], "A3": first fully connected layer's
    pre-activations [B][H]}.

    decisions (n = 1 only) replaces the network's own discrete choices by
    given ones, for tests that accept either outcome of a choice taken within
    rounding: "code1" [B][20][12][12] and "code2" [B][50][4][4] name each
    window's passing entry, "on1", "on2" (same shapes) and "on3" [B][H] say
    which ReLUs pass.  The network is then the same composition with those
    selections fixed (a pooled value is the named entry of its window)."""
    n, B, d = Xt.shape
    dcs = decisions or {}
    assert not dcs or n == 1
    assert d == CNN_IMG * CNN_IMG
    Wc1, bc1, Wc2, bc2, Wf1, bf1, Wf2, bf2 = cnn_split(w, H, C)
    G = np.empty((n, w.size))
    loss = np.empty(n)
    dec = [] if return_preact else None
    for i in range(n):
        X = np.asarray(Xt[i], dtype=np.float64).reshape(B, 1, CNN_IMG, CNN_IMG)
        y = np.asarray(yt[i], dtype=np.int64)
        Z1, cols1 = conv_valid(X, Wc1, bc1)                  # [B][20][24][24]
        P1, code1 = maxpool2(Z1)                             # [B][20][12][12]
        if "code1" in dcs:
            code1 = dcs["code1"]
            P1 = pool_take(Z1, code1)
        on1 = dcs.get("on1", P1 > 0.0)
        H1 = np.where(on1, P1, 0.0)
        Z2, cols2 = conv_valid(H1, Wc2, bc2)                 # [B][50][8][8]
        P2, code2 = maxpool2(Z2)                             # [B][50][4][4]
        if "code2" in dcs:
            code2 = dcs["code2"]
            P2 = pool_take(Z2, code2)
        on2 = dcs.get("on2", P2 > 0.0)
        H2 = np.where(on2, P2, 0.0)
        F = H2.reshape(B, CNN_FEAT)
        A3 = F @ Wf1 + bf1
        on3 = dcs.get("on3", A3 > 0.0)
        H3 = np.where(on3, A3, 0.0)
        Pr, ce = _softmax_ce(H3 @ Wf2 + bf2, y)
        R = (Pr - _onehot(y, C)) / B
        dWf2 = H3.T @ R
        dbf2 = R.sum(axis=0)
        dA3 = (R @ Wf2.T) * on3
        dWf1 = F.T @ dA3
        dbf1 = dA3.sum(axis=0)
        dH2 = (dA3 @ Wf1.T).reshape(P2.shape)
        dZ2 = maxpool2_grad(dH2 * on2, code2)
        dWc2 = conv_weight_grad(dZ2, cols2, Wc2.shape)
        dbc2 = dZ2.sum(axis=(0, 2, 3))
        dH1 = conv_input_grad(dZ2, Wc2, P1.shape[2], P1.shape[3])
        dZ1 = maxpool2_grad(dH1 * on1, code1)
        dWc1 = conv_weight_grad(dZ1, cols1, Wc1.shape)
        dbc1 = dZ1.sum(axis=(0, 2, 3))
        G[i] = np.concatenate([dWf1.ravel(), dbf1, dWf2.ravel(), dbf2,
                               dWc1.ravel(), dbc1, dWc2.ravel(), dbc2])
        loss[i] = ce.mean()
        if return_preact:
            dec.append({"Z1": Z1, "Z2": Z2, "A3": A3})
    if return_preact:
        return G, loss, dec
    return G, loss


def worker_grads(cfg, w, Xt, yt):
    """Dispatch on the workload's model."""
    if cfg.model == "softmax":
        return softmax_worker_grads(w, Xt, yt, cfg.C)
    if cfg.model == "cnn":
        return cnn_worker_grads(w, Xt, yt, cfg.H, cfg.C)
    return mlp_worker_grads(w, Xt, yt, cfg.H, cfg.C)
