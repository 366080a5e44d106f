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


def mlp_inputs(rng, n, B, d, H, C):
    X = rng.random((n, B, d), dtype=np.float32)
    y = rng.integers(0, C, size=(n, B), dtype=np.int32)
    W1 = (rng.standard_normal((d, H)) * np.sqrt(2.0 / d)).astype(np.float32)
    b1 = (0.01 * rng.standard_normal(H)).astype(np.float32)
    W2 = (rng.standard_normal((H, C)) * np.sqrt(2.0 / H)).astype(np.float32)
    b2 = (0.01 * rng.standard_normal(C)).astype(np.float32)
    w = np.concatenate([W1.ravel(), b1, W2.ravel(), b2])
    return X, y, w


def mlp_decision_flips(A_i, tau):
    """The hidden ReLUs of one worker (pre-activations A_i [B][H]) that fp32
    rounding could decide the other way: |A| < tau, with tau = frac x the
    largest |A| (frac 1e-6 is about 50x the rounding of a 784-term fp32 dot
    product).  Returns [(row, unit, other decision)]."""
    return [(int(b), int(u), not bool(A_i[b, u] > 0)) for b, u in np.argwhere(np.abs(A_i) < tau)]


def mlp_flip_deltas(w, X, y, H, C, A_i, flips):
    """Per flip, the oracle's change of the worker gradient (mean over its B
    rows) when that ReLU goes the other way: the flip's row alone, all its
    other units as the network's own.  X [B][d], y [B].  Returns [(unit,
    delta)]."""
    from oracle import model as omodel

    B = X.shape[0]
    w = np.asarray(w, dtype=np.float64)
    out = []
    for b, u, val in flips:
        own = {"on": A_i[b:b + 1] > 0}
        alt = {"on": own["on"].copy()}
        alt["on"][0, u] = val
        g0 = omodel.mlp_worker_grads(w, X[b][None, None], y[b][None, None], H, C, decisions=own)[0][0]
        g1 = omodel.mlp_worker_grads(w, X[b][None, None], y[b][None, None], H, C, decisions=alt)[0][0]
        out.append((u, (g1 - g0) / B))
    return out


def mlp_best_flip(a, o, deltas, d, H, C, limit=10):
    """o' = o plus, unit by unit, the subset of that unit's flip deltas that
    best matches a on the unit's column of dW1 and its b1 entry (where a flip
    acts; its effect elsewhere is of the order of the pre-activation, i.e.
    rounding).  Returns (largest per-block relative error over dW1, db1, dW2,
    db2, o')."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(o, dtype=np.float64).copy()
    by_unit = {}
    for u, dl in deltas:
        by_unit.setdefault(u, []).append(dl)
    for u, ds in by_unit.items():
        assert len(ds) <= limit, (u, len(ds))
        idx = np.r_[np.arange(u, d * H, H), d * H + u]
        best, pick = np.inf, None
        for m in range(1 << len(ds)):
            cand = ref[idx] + sum((dl[idx] for i, dl in enumerate(ds) if m >> i & 1), np.zeros(idx.size))
            err = float(np.max(np.abs(a[idx] - cand)))
            if err < best:
                best, pick = err, m
        for i, dl in enumerate(ds):
            if pick >> i & 1:
                ref += dl
    bounds = np.cumsum([0, d * H, H, H * C, C])
    err = max(float(np.max(np.abs(a[lo:hi] - ref[lo:hi]))) / max(float(np.max(np.abs(ref[lo:hi]))), 1e-30)
              for lo, hi in zip(bounds[:-1], bounds[1:]))
    return err, ref


def cnn_blocks(H, C):
    """[start, end) of the CNN's parameter blocks in G: Wf1, bf1, Wf2, bf2,
    Wc1, bc1, Wc2, bc2."""
    b = np.cumsum([0, 800 * H, H, H * C, C, 500, 20, 25000, 50])
    return list(zip(b[:-1], b[1:]))


def cnn_decision_flips(dec, frac=1e-6, conv_frac=2e-7):
    """The choices of one worker's network that fp32 rounding could take the
    other way, from the oracle's fp64 values (cnn_worker_grads with
    return_preact): another entry of a pooling window within conv_frac x the
    layer's largest magnitude of the window's largest (exactly equal entries
    are decided alike on both sides and are not listed), a pooled value that
    close to zero (its ReLU), a first fully connected unit with |A3| below
    frac x max|A3|.  Returns [(image, key, index, other choice)] with the keys
    of cnn_worker_grads' decisions."""
    from oracle import model as omodel

    out = []
    for layer, Z in ((1, dec["Z1"]), (2, dec["Z2"])):
        tol = conv_frac * float(np.max(np.abs(Z)))
        win = np.stack([Z[:, :, 0::2, 0::2], Z[:, :, 0::2, 1::2], Z[:, :, 1::2, 0::2], Z[:, :, 1::2, 1::2]])
        P, _ = omodel.maxpool2(Z)
        for a, b, o, py, px in np.argwhere((P[None] - win <= tol) & (win != P[None])):
            out.append((int(b), f"code{layer}", (int(o), int(py), int(px)), int(a)))
        for b, o, py, px in np.argwhere(np.abs(P) <= tol):
            out.append((int(b), f"on{layer}", (int(o), int(py), int(px)), not bool(P[b, o, py, px] > 0)))
    A = dec["A3"]
    for b, u in np.argwhere(np.abs(A) < frac * float(np.max(np.abs(A)))):
        out.append((int(b), "on3", (int(u),), not bool(A[b, u] > 0)))
    return out


def cnn_flip_deltas(w, X, y, H, C, dec, flips):
    """Per flip, the oracle's change of the worker gradient (the mean over its
    B images) when that one choice goes the other way: the flip's image
    alone, run with all its other choices as the network's own.  X [B][784],
    y [B]."""
    from oracle import model as omodel

    B = X.shape[0]
    w = np.asarray(w, dtype=np.float64)
    base, deltas = {}, []
    for b, key, idx, val in flips:
        if b not in base:
            P1, c1 = omodel.maxpool2(dec["Z1"][b:b + 1])
            P2, c2 = omodel.maxpool2(dec["Z2"][b:b + 1])
            own = {"code1": c1, "on1": P1 > 0, "code2": c2, "on2": P2 > 0, "on3": dec["A3"][b:b + 1] > 0}
            g = omodel.cnn_worker_grads(w, X[b][None, None], y[b][None, None], H, C, decisions=own)[0][0]
            base[b] = (own, g)
        own, g0 = base[b]
        alt = dict(own)
        alt[key] = own[key].copy()
        alt[key][(0, *idx)] = val
        g = omodel.cnn_worker_grads(w, X[b][None, None], y[b][None, None], H, C, decisions=alt)[0][0]
        if np.any(g != g0):
            deltas.append((g - g0) / B)
    return deltas


def cnn_best_flip(a, o, deltas, H, C, limit=12):
    """o' = o plus the sum of the subset of the flips' deltas (each choice
    within rounding may go either way) that minimises the largest per-block
    relative error max|a - o'| / max|o'| over the CNN's parameter blocks.
    Returns (that error, o')."""
    assert len(deltas) <= limit, len(deltas)
    a = np.asarray(a, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    best, best_ref = np.inf, o
    for m in range(1 << len(deltas)):
        ref = o.copy()
        for i, d in enumerate(deltas):
            if m >> i & 1:
                ref += d
        err = max(float(np.max(np.abs(a[lo:hi] - ref[lo:hi]))) / max(float(np.max(np.abs(ref[lo:hi]))), 1e-30)
                  for lo, hi in cnn_blocks(H, C))
        if err < best:
            best, best_ref = err, ref
    return best, best_ref


def cnn_best_flip_err(a, o, deltas, H, C, limit=12) -> float:
    """The error of cnn_best_flip."""
    return cnn_best_flip(a, o, deltas, H, C, limit)[0]
