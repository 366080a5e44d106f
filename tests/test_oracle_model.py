"""Pins of the oracle's worker gradients (Sect. 2, Eq. gradient) against
facts that do not come from the oracle's own formulas: finite differences of
the loss, the closed form at W = 0, autograd, the softmax row-sum identity and
the union-batch invariant of full synchronisation."""
import numpy as np
import pytest

from oracle import model, ps


def _mean_ce_softmax(w, X, y, C):
    W = w.reshape(X.shape[1], C)
    Z = X @ W
    Z = Z - Z.max(axis=1, keepdims=True)
    logp = Z - np.log(np.exp(Z).sum(axis=1, keepdims=True))
    return -logp[np.arange(len(y)), y].mean()


def _mean_ce_mlp(w, X, y, H, C):
    d = X.shape[1]
    W1 = w[:d * H].reshape(d, H)
    b1 = w[d * H:d * H + H]
    W2 = w[d * H + H:d * H + H + H * C].reshape(H, C)
    b2 = w[d * H + H + H * C:]
    Z = np.maximum(X @ W1 + b1, 0.0) @ W2 + b2
    Z = Z - Z.max(axis=1, keepdims=True)
    logp = Z - np.log(np.exp(Z).sum(axis=1, keepdims=True))
    return -logp[np.arange(len(y)), y].mean()


def _central_diff(f, w, h=1e-6):
    g = np.empty_like(w)
    for p in range(w.size):
        e = np.zeros_like(w)
        e[p] = h
        g[p] = (f(w + e) - f(w - e)) / (2 * h)
    return g


def test_softmax_finite_differences():
    rng = np.random.default_rng(1)
    n, B, d, C = 2, 3, 5, 4
    Xt = rng.normal(size=(n, B, d))
    yt = rng.integers(0, C, size=(n, B))
    w = rng.normal(scale=0.5, size=d * C)
    G, loss = model.softmax_worker_grads(w, Xt, yt, C)
    for i in range(n):
        fd = _central_diff(lambda v: _mean_ce_softmax(v, Xt[i], yt[i], C), w)
        assert np.max(np.abs(G[i] - fd)) <= 1e-7 * max(1.0, np.max(np.abs(fd)))
        assert loss[i] == pytest.approx(_mean_ce_softmax(w, Xt[i], yt[i], C), rel=1e-12)


def test_softmax_closed_form_at_zero():
    rng = np.random.default_rng(2)
    n, B, d, C = 3, 7, 6, 5
    Xt = rng.random((n, B, d))
    yt = rng.integers(0, C, size=(n, B))
    G, loss = model.softmax_worker_grads(np.zeros(d * C), Xt, yt, C)
    for i in range(n):
        Y = np.eye(C)[yt[i]]
        expect = Xt[i].T @ (np.full((B, C), 1.0 / C) - Y) / B
        np.testing.assert_allclose(G[i].reshape(d, C), expect, rtol=0, atol=1e-15)
        assert loss[i] == pytest.approx(np.log(C), rel=1e-14)


def test_softmax_rows_sum_to_zero_over_classes():
    # sum_c (P - Y)_{bc} = 0, so every feature's gradient sums to 0 over classes.
    rng = np.random.default_rng(3)
    n, B, d, C = 2, 9, 11, 7
    Xt = rng.normal(size=(n, B, d))
    yt = rng.integers(0, C, size=(n, B))
    G, _ = model.softmax_worker_grads(rng.normal(size=d * C), Xt, yt, C)
    assert np.max(np.abs(G.reshape(n, d, C).sum(axis=2))) < 1e-13


def test_softmax_matches_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(4)
    n, B, d, C = 3, 16, 20, 10
    Xt = rng.normal(size=(n, B, d))
    yt = rng.integers(0, C, size=(n, B))
    w = rng.normal(scale=0.1, size=d * C)
    G, loss = model.softmax_worker_grads(w, Xt, yt, C)
    for i in range(n):
        W = torch.tensor(w.reshape(d, C), dtype=torch.float64, requires_grad=True)
        L = torch.nn.functional.cross_entropy(torch.tensor(Xt[i]) @ W, torch.tensor(yt[i]))
        L.backward()
        np.testing.assert_allclose(G[i], W.grad.numpy().ravel(), rtol=1e-12, atol=1e-14)
        assert loss[i] == pytest.approx(L.item(), rel=1e-12)


def test_mlp_finite_differences():
    rng = np.random.default_rng(5)
    n, B, d, H, C = 2, 3, 5, 4, 3
    Xt = rng.normal(size=(n, B, d))
    yt = rng.integers(0, C, size=(n, B))
    w = rng.normal(scale=0.7, size=d * H + H + H * C + C)
    G, loss, A = model.mlp_worker_grads(w, Xt, yt, H, C, return_preact=True)
    assert np.min(np.abs(A)) > 1e-3  # away from ReLU kinks, so differences are valid
    for i in range(n):
        fd = _central_diff(lambda v: _mean_ce_mlp(v, Xt[i], yt[i], H, C), w)
        assert np.max(np.abs(G[i] - fd)) <= 1e-7 * max(1.0, np.max(np.abs(fd)))
        assert loss[i] == pytest.approx(_mean_ce_mlp(w, Xt[i], yt[i], H, C), rel=1e-12)


def test_mlp_matches_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(6)
    n, B, d, H, C = 2, 8, 12, 16, 10
    Xt = rng.random((n, B, d))
    yt = rng.integers(0, C, size=(n, B))
    w = rng.normal(scale=0.3, size=d * H + H + H * C + C)
    G, loss = model.mlp_worker_grads(w, Xt, yt, H, C)
    for i in range(n):
        W1 = torch.tensor(w[:d * H].reshape(d, H), requires_grad=True)
        b1 = torch.tensor(w[d * H:d * H + H], requires_grad=True)
        W2 = torch.tensor(w[d * H + H:d * H + H + H * C].reshape(H, C), requires_grad=True)
        b2 = torch.tensor(w[d * H + H + H * C:], requires_grad=True)
        Z = torch.relu(torch.tensor(Xt[i]) @ W1 + b1) @ W2 + b2
        L = torch.nn.functional.cross_entropy(Z, torch.tensor(yt[i]))
        L.backward()
        ref = np.concatenate([W1.grad.numpy().ravel(), b1.grad.numpy(),
                              W2.grad.numpy().ravel(), b2.grad.numpy()])
        np.testing.assert_allclose(G[i], ref, rtol=1e-11, atol=1e-14)
        assert loss[i] == pytest.approx(L.item(), rel=1e-12)


@pytest.mark.parametrize("which", ["softmax", "mlp"])
def test_full_sync_equals_union_batch(which):
    # Averaging all n workers' gradients equals the gradient on the union of
    # their minibatches (n*B rows), because every worker uses the same w_t.
    rng = np.random.default_rng(7)
    n, B, d, H, C = 5, 6, 9, 7, 4
    Xt = rng.normal(size=(n, B, d))
    yt = rng.integers(0, C, size=(n, B))
    if which == "softmax":
        w = rng.normal(scale=0.3, size=d * C)
        G, loss = model.softmax_worker_grads(w, Xt, yt, C)
        Gu, lu = model.softmax_worker_grads(w, Xt.reshape(1, n * B, d), yt.reshape(1, n * B), C)
    else:
        w = rng.normal(scale=0.3, size=d * H + H + H * C + C)
        G, loss = model.mlp_worker_grads(w, Xt, yt, H, C)
        Gu, lu = model.mlp_worker_grads(w, Xt.reshape(1, n * B, d), yt.reshape(1, n * B), H, C)
    g = ps.aggregate(G, list(range(n)))
    np.testing.assert_allclose(g, Gu[0], rtol=1e-12, atol=1e-15)
    assert np.mean(loss) == pytest.approx(lu[0], rel=1e-12)
