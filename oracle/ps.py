"""Parameter-server side of one iteration, float64.

* select_fastest -- the PS uses the first k gradients to arrive (Sect. 2,
  Eq. grad_bw).  Arrival order is the order of the round-trip ticks; equal
  ticks are broken toward the lower worker index.
* aggregate      -- g_t = (1/k) sum over the k received gradients (Eq. grad_bw).
* grad_stats     -- end-of-iteration estimators (Sect. 3.1):
    V+  = sum_l (1/(k-1)) sum_j ([g_j - g_t]_l)^2          (Eq. sumvariancekt)
    N+  = max(||g_t||^2 - V+/k, 0)                          (Eq. normsquarekt)
    F^  = mean of the received workers' minibatch losses   (loss estimate)
  With k = 1 the unbiased variance estimator is undefined; V+ then takes the
  current D-window average of past V+ values (0 without history).
* sgd_update     -- w_{t+1} = w_t - eta g_t (Eq. update).

Test infrastructure only (see the package docstring).
"""
from __future__ import annotations

import numpy as np


def select_fastest(ticks, k: int):
    """Return (sel, mask): sel = the k workers with the smallest
    (tick, index) pairs, listed in arrival order; mask[i] = 1 iff i in sel."""
    ticks = [int(x) for x in ticks]
    n = len(ticks)
    if not 1 <= k <= n:
        raise ValueError(f"k={k} outside [1, {n}]")
    order = sorted(range(n), key=lambda i: (ticks[i], i))
    sel = order[:k]
    mask = np.zeros(n, dtype=np.uint8)
    mask[sel] = 1
    return sel, mask


def aggregate(G: np.ndarray, sel) -> np.ndarray:
    """Average of the selected rows of G (float64)."""
    rows = np.asarray(G, dtype=np.float64)[list(sel)]
    return rows.sum(axis=0) / len(sel)


def grad_stats(G: np.ndarray, sel, g: np.ndarray, loss, V_window: float = 0.0):
    """End-of-iteration statistics over the k received gradients.

    Returns a dict with sqnorm [n] (||g_j||^2 for received j, 0 otherwise),
    gnorm2 = ||g_t||^2, V_plus, N_plus and F_hat.
    """
    G = np.asarray(G, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    sel = list(sel)
    k = len(sel)
    n = G.shape[0]
    sqnorm = np.zeros(n)
    for j in sel:
        sqnorm[j] = float(np.dot(G[j], G[j]))
    gnorm2 = float(np.dot(g, g))
    if k >= 2:
        dev = G[sel] - g[None, :]
        V_plus = float((dev * dev).sum()) / (k - 1)
    else:
        V_plus = float(V_window)
    N_plus = max(gnorm2 - V_plus / k, 0.0)
    F_hat = float(np.mean(np.asarray(loss, dtype=np.float64)[sel]))
    return {"sqnorm": sqnorm, "gnorm2": gnorm2, "V_plus": V_plus,
            "N_plus": N_plus, "F_hat": F_hat}


def sgd_update(w: np.ndarray, g: np.ndarray, eta: float) -> np.ndarray:
    return np.asarray(w, dtype=np.float64) - eta * np.asarray(g, dtype=np.float64)
