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


# -- the CNN -----------------------------------------------------------------

def _cnn_torch(w, X, y, H, C, torch):
    """The network from its layer definitions in torch (float64, CPU)."""
    F = torch.nn.functional
    sizes = [(800, H), (H,), (H, C), (C,), (20, 1, 5, 5), (20,), (50, 20, 5, 5), (50,)]
    ps_, o = [], 0
    for sh in sizes:
        m = int(np.prod(sh))
        ps_.append(torch.tensor(w[o:o + m].reshape(sh), requires_grad=True))
        o += m
    Wf1, bf1, Wf2, bf2, Wc1, bc1, Wc2, bc2 = ps_
    x = torch.tensor(X.reshape(-1, 1, 28, 28))
    a = F.relu(F.max_pool2d(F.conv2d(x, Wc1, bc1), 2))
    a = F.relu(F.max_pool2d(F.conv2d(a, Wc2, bc2), 2))
    a = F.relu(a.reshape(-1, 800) @ Wf1 + bf1)
    L = F.cross_entropy(a @ Wf2 + bf2, torch.tensor(y))
    L.backward()
    return np.concatenate([p.grad.numpy().ravel() for p in ps_]), L.item()


def test_cnn_matches_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(61)
    n, B, H, C = 2, 5, 24, 10
    Xt = np.where(rng.random((n, B, 784)) < 0.7, 0.0, rng.random((n, B, 784)))
    yt = rng.integers(0, C, size=(n, B))
    w = rng.uniform(-0.3, 0.3, size=model.cnn_param_count(H, C))
    G, loss = model.cnn_worker_grads(w, Xt, yt, H, C)
    for i in range(n):
        ref, L = _cnn_torch(w, Xt[i], yt[i], H, C, torch)
        np.testing.assert_allclose(G[i], ref, rtol=1e-10, atol=1e-13)
        assert loss[i] == pytest.approx(L, rel=1e-12)


def test_cnn_finite_differences():
    # a few parameters of every block, one worker of three images
    rng = np.random.default_rng(62)
    B, H, C = 3, 8, 4
    X = rng.random((1, B, 784))
    y = rng.integers(0, C, size=(1, B))
    w = rng.uniform(-0.15, 0.15, size=model.cnn_param_count(H, C))
    G, L0 = model.cnn_worker_grads(w, X, y, H, C)

    def loss_at(v):
        return model.cnn_worker_grads(v, X, y, H, C)[1][0]

    bounds = np.cumsum([0, 800 * H, H, H * C, C, 500, 20, 25000, 50])
    for lo, hi in zip(bounds[:-1], bounds[1:]):
        for p in rng.choice(np.arange(lo, hi), size=min(4, hi - lo), replace=False):
            # a step that crosses a ReLU or pooling decision shows as one-sided
            # differences that disagree: then a smaller step
            for h in (1e-5, 1e-6, 1e-7):
                e = np.zeros_like(w)
                e[p] = h
                lp, lm = loss_at(w + e), loss_at(w - e)
                tol = 50 * 2.2e-16 * L0[0] / h        # rounding of the losses
                if abs((lp - L0[0]) - (L0[0] - lm)) / h <= 1e-3 * abs(lp - lm) / (2 * h) + 4 * tol:
                    break
            fd = (lp - lm) / (2 * h)
            assert G[0, p] == pytest.approx(fd, rel=1e-4, abs=tol), (lo, p, h)


def test_mlp_fixed_decisions_match_finite_differences():
    # With the ReLUs fixed (some flipped from the network's own), the loss is
    # smooth in w and the oracle returns its gradient; its own decisions,
    # passed in, change nothing; a flip moves its unit's W1 column and b1.
    rng = np.random.default_rng(67)
    B, d, H, C = 3, 12, 9, 4
    X = rng.normal(size=(1, B, d))
    y = rng.integers(0, C, size=(1, B))
    w = rng.normal(size=d * H + H + H * C + C) * 0.4
    G0, L0, A = model.mlp_worker_grads(w, X, y, H, C, return_preact=True)
    own = {"on": A[0] > 0}
    G1, L1 = model.mlp_worker_grads(w, X, y, H, C, decisions=own)
    np.testing.assert_array_equal(G1, G0)
    assert L1[0] == L0[0]
    flip = {"on": own["on"].copy()}
    flip["on"][1, 4] = ~flip["on"][1, 4]
    flip["on"][2, 7] = ~flip["on"][2, 7]
    G, _ = model.mlp_worker_grads(w, X, y, H, C, decisions=flip)
    assert not np.array_equal(G[0, 4:d * H:H], G0[0, 4:d * H:H])
    assert G[0, d * H + 7] != G0[0, d * H + 7]

    def loss_at(v):
        return model.mlp_worker_grads(v, X, y, H, C, decisions=flip)[1][0]

    h = 1e-6
    for p in range(w.size):
        e = np.zeros_like(w)
        e[p] = h
        fd = (loss_at(w + e) - loss_at(w - e)) / (2 * h)
        assert G[0, p] == pytest.approx(fd, rel=1e-5, abs=1e-9), p


def test_cnn_fixed_decisions_match_finite_differences():
    # With every pooling choice and ReLU fixed (some of them flipped from the
    # network's own), the loss is a smooth function of w whose gradient the
    # oracle must return; and its own decisions, passed in, change nothing.
    rng = np.random.default_rng(65)
    B, H, C = 2, 8, 4
    X = rng.random((1, B, 784))
    y = rng.integers(0, C, size=(1, B))
    w = rng.uniform(-0.15, 0.15, size=model.cnn_param_count(H, C))
    G0, L0, dec = model.cnn_worker_grads(w, X, y, H, C, return_preact=True)
    Z1, Z2, A3 = dec[0]["Z1"], dec[0]["Z2"], dec[0]["A3"]
    P1, code1 = model.maxpool2(Z1)
    P2, code2 = model.maxpool2(Z2)
    own = {"code1": code1, "on1": P1 > 0, "code2": code2, "on2": P2 > 0, "on3": A3 > 0}
    G1, L1 = model.cnn_worker_grads(w, X, y, H, C, decisions=own)
    np.testing.assert_array_equal(G1, G0)
    assert L1[0] == L0[0]
    flip = {k: v.copy() for k, v in own.items()}
    flip["code1"][0, 3, 5, 6] = (code1[0, 3, 5, 6] + 1) % 4
    flip["on1"][1, 7, 2, 2] = ~own["on1"][1, 7, 2, 2]
    j = np.argwhere(own["on2"][0])[0]                  # a passing conv2 window
    flip["code2"][0][tuple(j)] = (code2[0][tuple(j)] + 2) % 4
    flip["on2"][1, 10, 1, 3] = ~own["on2"][1, 10, 1, 3]
    flip["on3"][0, 2] = ~own["on3"][0, 2]
    G, L = model.cnn_worker_grads(w, X, y, H, C, decisions=flip)
    bounds = np.cumsum([0, 800 * H, H, H * C, C, 500, 20, 25000, 50])
    # each override on its own moves the gradient where it must
    for key, idx, lo, hi in (("code1", (0, 3, 5, 6), bounds[4] + 75, bounds[4] + 100),
                             ("on1", (1, 7, 2, 2), bounds[4] + 175, bounds[4] + 200),
                             ("code2", (0, *j), bounds[6] + j[0] * 500, bounds[6] + j[0] * 500 + 500),
                             ("on2", (1, 10, 1, 3), bounds[7] + 10, bounds[7] + 11),
                             ("on3", (0, 2), bounds[1] + 2, bounds[1] + 3)):
        one = dict(own)
        one[key] = own[key].copy()
        one[key][idx] = flip[key][idx]
        Gk = model.cnn_worker_grads(w, X, y, H, C, decisions=one)[0]
        assert not np.array_equal(Gk[0, lo:hi], G0[0, lo:hi]), key

    def loss_at(v):
        return model.cnn_worker_grads(v, X, y, H, C, decisions=flip)[1][0]

    # every conv1 weight and every bias; in the large blocks random entries
    # plus those the flips touch (conv2 filter j[0], the first layer's unit 2)
    check = [np.arange(bounds[4], bounds[6]), np.arange(bounds[7], bounds[8]),
             np.arange(bounds[1], bounds[2]), np.arange(bounds[3], bounds[4]),
             rng.choice(np.arange(bounds[0], bounds[1]), 12, replace=False),
             np.arange(2, 800 * H, H)[rng.choice(800, 12, replace=False)],
             rng.choice(np.arange(bounds[2], bounds[3]), 12, replace=False),
             rng.choice(np.arange(bounds[6], bounds[7]), 12, replace=False),
             bounds[6] + j[0] * 500 + rng.choice(500, 24, replace=False)]
    h = 1e-5
    for p in np.concatenate(check):
        e = np.zeros_like(w)
        e[p] = h
        fd = (loss_at(w + e) - loss_at(w - e)) / (2 * h)
        assert G[0, p] == pytest.approx(fd, rel=1e-5, abs=1e-9), p


def test_cnn_closed_form_at_zero():
    # all parameters 0: logits 0, uniform class probabilities, loss ln C; only
    # the last bias has a gradient, the batch mean of 1/C - onehot(y)
    B, H, C = 6, 10, 5
    y = np.array([[0, 1, 1, 4, 2, 1]])
    X = np.random.default_rng(63).random((1, B, 784))
    G, loss = model.cnn_worker_grads(np.zeros(model.cnn_param_count(H, C)), X, y, H, C)
    expect = np.zeros(model.cnn_param_count(H, C))
    o = 800 * H + H + H * C          # the last bias
    expect[o:o + C] = [(1 / C) - np.mean(y[0] == c) for c in range(C)]
    np.testing.assert_allclose(G[0], expect, rtol=0, atol=1e-15)
    assert loss[0] == pytest.approx(np.log(C), rel=1e-14)


def test_convolution_and_its_input_gradient_by_loops():
    rng = np.random.default_rng(64)
    B, Ci, h, wd, Co, k = 2, 3, 6, 7, 4, 3
    X = rng.normal(size=(B, Ci, h, wd))
    W = rng.normal(size=(Co, Ci, k, k))
    b = rng.normal(size=Co)
    out, _ = model.conv_valid(X, W, b)
    dOut = rng.normal(size=out.shape)
    ref = np.zeros_like(out)
    dX = np.zeros_like(X)
    for bb in range(B):
        for o in range(Co):
            for y in range(h - k + 1):
                for x in range(wd - k + 1):
                    ref[bb, o, y, x] = b[o] + sum(X[bb, c, y + u, x + v] * W[o, c, u, v]
                                                  for c in range(Ci) for u in range(k) for v in range(k))
                    for c in range(Ci):
                        for u in range(k):
                            for v in range(k):
                                dX[bb, c, y + u, x + v] += dOut[bb, o, y, x] * W[o, c, u, v]
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(model.conv_input_grad(dOut, W, h, wd), dX, rtol=1e-12, atol=1e-12)


def test_pooling_passes_the_first_of_equal_values():
    Z = np.array([[[[1.0, 3.0, 2.0, 2.0],
                    [3.0, 0.0, 2.0, 2.0]]]])           # windows: (1,3,3,0) and (2,2,2,2)
    P, code = model.maxpool2(Z)
    assert P.tolist() == [[[[3.0, 2.0]]]] and code.tolist() == [[[[1, 0]]]]
    dZ = model.maxpool2_grad(np.array([[[[5.0, 7.0]]]]), code)
    assert dZ.tolist() == [[[[0.0, 5.0, 7.0, 0.0], [0.0, 0.0, 0.0, 0.0]]]]
