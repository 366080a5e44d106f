"""Helpers shared by the GPU tests: seeded inputs, error metrics, contexts."""
from __future__ import annotations

import numpy as np

RTOL = 1e-4   # max relative error for fp32 gradients and statistics


def rel_err(a, o) -> float:
    """max_l |a_l - o_l| / max_l |o_l| (arrays) -- the parity metric."""
    a = np.asarray(a, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    den = float(np.max(np.abs(o))) if o.size else 0.0
    num = float(np.max(np.abs(a - o))) if o.size else 0.0
    return num / max(den, 1e-30)


def scalar_rel(a, o) -> float:
    return abs(float(a) - float(o)) / max(abs(float(o)), 1e-30)


def softmax_inputs(rng, n, B, d, C, S=None, features="normal"):
    """Materialised minibatches (X [n][B][d], y [n][B]) and W [d*C], or with S
    a dataset [S][d], labels [S] and row indices [n][B]."""
    rows = S if S is not None else n * B
    if features == "normal":
        X = rng.standard_normal((rows, d), dtype=np.float32)
    else:
        X = rng.random((rows, d), dtype=np.float32)
    y = rng.integers(0, C, size=rows, dtype=np.int32)
    W = (0.05 * rng.standard_normal(d * C)).astype(np.float32)
    if S is None:
        return X.reshape(n, B, d), y.reshape(n, B), W, None
    idx = rng.integers(0, S, size=(n, B), dtype=np.int32)
    return X, y, W, idx


def to_dev(torch, a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def k_acceptable(objective, k_gpu: int, k_ref: int, tol: float = 1e-6) -> bool:
    """The chosen k matches, or the oracle's objective at k_gpu ties the best
    within tol (relative)."""
    if k_gpu == k_ref:
        return True
    if objective is None:
        return False
    vals = [v for v in objective if v is not None]
    if not vals:
        return False
    best = max(vals)
    v = objective[k_gpu - 1]
    return v is not None and v >= best - tol * abs(best)
