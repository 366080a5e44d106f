"""Pins of the oracle's PS-side arithmetic: fastest-k selection, averaging and
the end-of-iteration estimators (Sect. 2 Eq. grad_bw; Sect. 3.1 Eqs.
second_moment, sumvariancekt, normsquarekt, estimateL, exp_decrease).

The statistical pins draw minibatches with replacement from a tiny finite
set of per-sample gradients, where the true full gradient and the true
minibatch variance are known exactly."""
import itertools

import numpy as np
import pytest

from oracle import dbw, ps


# -- selection ---------------------------------------------------------------

def test_select_matches_brute_force_sort():
    rng = np.random.default_rng(11)
    for _ in range(200):
        n = int(rng.integers(1, 12))
        ticks = rng.integers(1, 6, size=n)       # many ties on purpose
        k = int(rng.integers(1, n + 1))
        sel, mask = ps.select_fastest(ticks, k)
        # brute force: worker i is selected iff fewer than k workers come
        # strictly before it in (tick, index) order
        for i in range(n):
            before = sum(1 for j in range(n) if (ticks[j], j) < (ticks[i], i))
            assert mask[i] == (1 if before < k else 0)
        assert len(sel) == k and sorted(sel) == sorted(np.flatnonzero(mask).tolist())


def test_select_ties_go_to_lower_index():
    sel, mask = ps.select_fastest([5, 3, 3, 3, 9], 2)
    assert sel == [1, 2] and mask.tolist() == [0, 1, 1, 0, 0]
    sel, _ = ps.select_fastest([7, 7, 7, 7], 3)
    assert sel == [0, 1, 2]
    with pytest.raises(ValueError):
        ps.select_fastest([1, 2], 0)
    with pytest.raises(ValueError):
        ps.select_fastest([1, 2], 3)


def test_k1_is_fastest_worker_and_permutation_invariance():
    rng = np.random.default_rng(12)
    n, P = 7, 13
    G = rng.normal(size=(n, P))
    ticks = rng.permutation(np.arange(10, 10 + n))
    sel, _ = ps.select_fastest(ticks, 1)
    np.testing.assert_array_equal(ps.aggregate(G, sel), G[int(np.argmin(ticks))])
    k = 4
    g = ps.aggregate(G, ps.select_fastest(ticks, k)[0])
    perm = rng.permutation(n)
    g2 = ps.aggregate(G[perm], ps.select_fastest(ticks[perm], k)[0])
    np.testing.assert_allclose(g, g2, rtol=1e-14)


# -- estimators: deterministic cases -------------------------------------------

def test_identical_gradients_have_zero_variance():
    g0 = np.array([0.5, -1.0, 2.0])
    G = np.tile(g0, (5, 1))
    sel = [0, 2, 3]
    st = ps.grad_stats(G, sel, ps.aggregate(G, sel), np.array([1, 2, 3, 4, 5.0]))
    assert st["V_plus"] == 0.0
    assert st["N_plus"] == pytest.approx(float(g0 @ g0), rel=1e-15)
    assert st["F_hat"] == pytest.approx((1 + 3 + 4) / 3, rel=1e-15)
    np.testing.assert_allclose(st["sqnorm"], [g0 @ g0, 0, g0 @ g0, g0 @ g0, 0])


def test_two_pass_variance_equals_moment_form():
    rng = np.random.default_rng(13)
    G = rng.normal(size=(9, 40))
    sel = [8, 1, 4, 6, 2]
    g = ps.aggregate(G, sel)
    st = ps.grad_stats(G, sel, g, np.zeros(9))
    k = len(sel)
    moment = (sum(G[j] @ G[j] for j in sel) - k * (g @ g)) / (k - 1)
    assert st["V_plus"] == pytest.approx(moment, rel=1e-12)
    # N+ clips at zero
    assert st["N_plus"] == max(g @ g - st["V_plus"] / k, 0.0)


def test_k1_uses_window_variance():
    G = np.arange(12.0).reshape(3, 4)
    st = ps.grad_stats(G, [2], G[2], np.ones(3), V_window=7.5)
    assert st["V_plus"] == 7.5
    assert st["N_plus"] == pytest.approx(max(G[2] @ G[2] - 7.5, 0.0))


# -- estimators: statistical pins ------------------------------------------------

def _finite_problem():
    # per-sample gradients u_l of a finite dataset (S = 6 points in R^3)
    u = np.array([[1.0, 0.2, -0.5], [0.4, -1.0, 0.3], [2.0, 0.5, 0.1],
                  [-0.3, 0.8, 1.2], [0.9, 0.0, -0.7], [1.5, -0.4, 0.6]])
    grad_F = u.mean(axis=0)
    return u, grad_F


def test_monte_carlo_second_moment_and_unbiased_variance():
    # Eq. second_moment: E||g_t||^2 = ||grad F||^2 + V/k, and Eq. sumvariancekt
    # is unbiased for V = Var of one worker's gradient (sum over components).
    u, grad_F = _finite_problem()
    S = u.shape[0]
    B, n, k = 2, 5, 3
    V_true = ((u - grad_F) ** 2).sum(axis=1).mean() / B   # with-replacement sampling
    rng = np.random.default_rng(14)
    reps = 20000
    gn, vp, nn = np.empty(reps), np.empty(reps), np.empty(reps)
    for r in range(reps):
        G = u[rng.integers(0, S, size=(n, B))].mean(axis=1)
        sel = [0, 1, 2]
        st = ps.grad_stats(G, sel, ps.aggregate(G, sel), np.zeros(n))
        gn[r], vp[r] = st["gnorm2"], st["V_plus"]
        nn[r] = st["gnorm2"] - st["V_plus"] / k
    se = lambda a: a.std(ddof=1) / np.sqrt(reps)
    assert abs(vp.mean() - V_true) < 5 * se(vp)
    assert abs(gn.mean() - (grad_F @ grad_F + V_true / k)) < 5 * se(gn)
    # ||g||^2 - V+/k is unbiased for ||grad F||^2 (Eq. normsquarekt before clipping)
    assert abs(nn.mean() - grad_F @ grad_F) < 5 * se(nn)


@pytest.mark.parametrize("k", [1, 2, 4])
def test_monte_carlo_gain_formula(k):
    # Eq. exp_decrease: E[eta gradF.g - L eta^2/2 ||g||^2] for the average of k
    # workers' gradients equals (eta - L eta^2/2)||gradF||^2 - (L eta^2/2) V/k.
    u, grad_F = _finite_problem()
    S = u.shape[0]
    B, eta, L = 3, 0.3, 2.5
    V_true = ((u - grad_F) ** 2).sum(axis=1).mean() / B
    rng = np.random.default_rng(15 + k)
    reps = 40000
    G = u[rng.integers(0, S, size=(reps, k, B))].mean(axis=2).mean(axis=1)
    samples = eta * (G @ grad_F) - L * eta ** 2 / 2 * (G * G).sum(axis=1)
    expect = dbw.gains(V_true, float(grad_F @ grad_F), L, eta, k)[k - 1]
    se = samples.std(ddof=1) / np.sqrt(reps)
    assert abs(samples.mean() - expect) < 5 * se


def test_l_estimate_exact_on_quadratic():
    # F(w) = a/2 ||w||^2 with exact gradients (no minibatch noise): the
    # smoothness estimate of Eq. estimateL recovers a exactly.
    for a, eta in [(0.7, 0.1), (3.0, 0.05), (1.0, 1.3)]:
        w_prev = np.array([1.0, -2.0, 0.5])
        grad = a * w_prev
        w_now = w_prev - eta * grad
        F = lambda w: 0.5 * a * (w @ w)
        N_prev = float(grad @ grad)
        L = dbw.l_estimate(eta, N_prev, 0.0, 4, F(w_prev), F(w_now))
        assert L == pytest.approx(a, rel=1e-12)
    assert dbw.l_estimate(0.1, 0.0, 0.0, 3, 1.0, 0.9) is None   # zero denominator


def test_sgd_update():
    w = np.array([1.0, 2.0])
    np.testing.assert_array_equal(ps.sgd_update(w, np.array([0.5, -1.0]), 0.1), [0.95, 2.1])


def test_window_mean():
    assert dbw.window_mean([], 5) is None
    assert dbw.window_mean([1.0, 2.0], 5) == 1.5
    assert dbw.window_mean([9.0, 1.0, 2.0, 3.0, 4.0, 5.0], 5) == 3.0
    for h in itertools.islice(itertools.count(1), 6):
        hist = list(range(h))
        assert dbw.window_mean([float(x) for x in hist], 3) == np.mean(hist[-3:])
