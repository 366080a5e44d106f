"""Pins of the oracle's choice of k (Sect. 3.3, Eqs. gain, greedy, greedy2)
and of its iteration bookkeeping."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from dbw_inputs import C1, SOFTMAX, DBWConfig, TimeModel, gather, init_params
from dbw_inputs import generate as gen
from oracle import dbw


def _choose(n, V, N, L, T_hat, eta=0.1, beta=1.01, F=(1.0, 1.0), k_prev=None):
    k_prev = n if k_prev is None else k_prev
    return dbw.choose_k(n, eta, beta, 5, [V], [N], [L], list(F), k_prev, T_hat)


def test_no_history_waits_for_all():
    k, obj = dbw.choose_k(6, 0.1, 1.01, 5, [1.0], [1.0], [], [1.0], 6, [1.0] * 6)
    assert k == 6 and obj is None


def test_zero_variance_picks_fastest_time_largest_tie():
    # V = 0: every gain equals (eta - L eta^2/2) N > 0, so the ratio is largest
    # where T_hat is smallest; among equal T_hat the largest k wins.
    k, _ = _choose(4, 0.0, 2.0, 1.0, [3.0, 2.0, 2.0, 5.0])
    assert k == 3


def test_all_gains_negative_waits_for_all():
    # N = 0, V > 0, L > 0: every gain is negative.
    k, obj = _choose(5, 4.0, 0.0, 2.0, [1.0, 2.0, 3.0, 4.0, 5.0])
    assert k == 5 and all(o < 0 for o in obj)


def test_negative_l_prefers_smallest_k():
    # L < 0 makes the gain positive and decreasing in k; with increasing
    # T_hat the ratio is largest at k = 1.
    k, _ = _choose(6, 3.0, 0.1, -5.0, [1.0, 1.5, 2.0, 2.5, 3.0, 3.5])
    assert k == 1


def test_scale_invariance():
    rng = np.random.default_rng(21)
    for _ in range(50):
        n = int(rng.integers(2, 9))
        T = np.sort(rng.uniform(1, 3, size=n)).tolist()
        V, N, L = rng.uniform(0.1, 2), rng.uniform(0.1, 2), rng.uniform(-1, 5)
        k1, _ = _choose(n, V, N, L, T)
        k2, _ = _choose(n, 4 * V, 4 * N, L, [7.0 * x for x in T])
        assert k1 == k2


def test_missing_time_estimate_is_not_eligible():
    k, obj = _choose(4, 0.0, 1.0, 0.0, [None, 2.0, None, 1.0])
    assert k == 4 and obj[0] is None


def test_guard_forces_larger_k_when_loss_rises():
    T = [1.0, 2.0, 3.0, 4.0, 5.0, 6.0]
    base, _ = _choose(6, 3.0, 0.1, -5.0, T, F=(1.0, 1.0), k_prev=3)
    assert base == 1
    k, _ = _choose(6, 3.0, 0.1, -5.0, T, F=(1.0, 1.02), k_prev=3)   # 1.02 > 1.01 * 1.0
    assert k == 4
    k, _ = _choose(6, 3.0, 0.1, -5.0, T, F=(1.0, 1.005), k_prev=3)  # below beta
    assert k == 1
    k, _ = _choose(6, 3.0, 0.1, -5.0, T, F=(1.0, 1.02), k_prev=6)   # already n
    assert k == 1
    # the guard never lowers k
    k, _ = _choose(6, 0.0, 1.0, 1.0, [6, 5, 4, 3, 2, 1.0], F=(1.0, 2.0), k_prev=2)
    assert k == 6


def test_choice_maximises_exact_expected_decrease_per_time():
    # Gain by exhaustive enumeration: a finite problem with S = 3 per-sample
    # gradients, B = 1, k workers drawing with replacement.  The expectation in
    # Eq. gain_with_E is computed exactly over all S^k outcomes; dividing by
    # T_k and taking the argmax (largest k on ties) must give the oracle's k.
    u = [(Fraction(3), Fraction(-1)), (Fraction(1), Fraction(2)), (Fraction(-1), Fraction(1))]
    S = len(u)
    gF = tuple(sum(x[c] for x in u) / S for c in range(2))
    V = sum(sum((x[c] - gF[c]) ** 2 for c in range(2)) for x in u) / S   # B = 1
    N = sum(c * c for c in gF)
    n = 4
    for eta, L, T in [(Fraction(1, 10), Fraction(3), [1, 1.3, 1.5, 2.6]),
                      (Fraction(1, 2), Fraction(1), [1, 1.9, 2.1, 2.2]),
                      (Fraction(1, 5), Fraction(-2), [1, 1.1, 1.2, 1.3]),
                      (Fraction(1, 10), Fraction(20), [1, 2, 3, 4])]:
        exact = []
        for k in range(1, n + 1):
            tot = Fraction(0)
            for draw in itertools.product(range(S), repeat=k):
                g = tuple(sum(u[j][c] for j in draw) / k for c in range(2))
                tot += eta * (gF[0] * g[0] + gF[1] * g[1]) - L * eta * eta / 2 * (g[0] ** 2 + g[1] ** 2)
            exact.append(tot / S ** k)
        ratios = [exact[k] / Fraction(T[k]) for k in range(n)]
        if max(exact) < 0:
            expect = n
        else:
            best = max(ratios)
            expect = max(k + 1 for k in range(n) if ratios[k] == best)
        k, _ = dbw.choose_k(n, float(eta), 1.01, 5, [float(V)], [float(N)], [float(L)],
                            [1.0], n, T)
        assert k == expect


def _tiny_cfg(**kw):
    base = DBWConfig(name="tiny", model=SOFTMAX, n=4, B=8, d=12, C=3, S=200, iters=12,
                     features="uniform", times=TimeModel(kind="shifted_exp", shift=1.0, rate=1.0),
                     seed=777)
    return base.replace(**kw)


def test_trajectory_bookkeeping():
    cfg = _tiny_cfg()
    X, y = gen.dataset(cfg)
    orc = dbw.DBWOracle(cfg, init_params(cfg))
    clock = 0
    for t in range(cfg.iters):
        Xt, yt = gather(X, y, gen.batch_indices(cfg, t))
        ticks = gen.round_trip_ticks(cfg, t)
        h = orc.k_prev
        before = [row[:] for row in orc.cnt]
        rec = orc.step(Xt, yt, ticks)
        if t < 2:
            assert rec["k"] == cfg.n and rec["objective"] is None
        if t == 0:
            assert rec["T_hat"] == [None] * cfg.n
        else:
            assert all(x is not None and x > 0 for x in rec["T_hat"])
        # the n samples of iteration t land in row k_{t-1}
        assert orc.cnt[h - 1] == [c + 1 for c in before[h - 1]]
        clock += int(np.sort(ticks)[rec["k"] - 1])
        assert orc.clock == clock
        assert rec["b"] == cfg.n - rec["k"]
        assert len(orc.hV) == t + 1 and len(orc.hL) <= t
    st = orc.export_state()
    assert len(st["hV"]) == min(cfg.D, cfg.iters)


def test_static_full_sync_is_plain_sgd():
    # With k forced to n the trajectory is synchronous SGD on the union batch.
    cfg = _tiny_cfg()
    X, y = gen.dataset(cfg)
    orc = dbw.DBWOracle(cfg, init_params(cfg))
    w = init_params(cfg).astype(np.float64)
    from oracle import model
    for t in range(4):
        idx = gen.batch_indices(cfg, t)
        Xt, yt = gather(X, y, idx)
        orc.step(Xt, yt, gen.round_trip_ticks(cfg, t), k_force=cfg.n)
        Gu, _ = model.softmax_worker_grads(w, Xt.reshape(1, -1, cfg.d), yt.reshape(1, -1), cfg.C)
        w = w - cfg.eta * Gu[0]
        np.testing.assert_allclose(orc.w, w, rtol=1e-12, atol=1e-15)


def _choose_policy(n, V, N, L, T_hat, policy, k_static=0, F=(1.0, 1.0), k_prev=None, hL=True):
    k_prev = n if k_prev is None else k_prev
    return dbw.choose_k(n, 0.1, 1.01, 5, [V], [N], [L] if hL else [], list(F), k_prev, T_hat,
                        policy=policy, k_static=k_static)


def test_blind_gain_is_k_per_unit_time():
    # B-DBW: objective k / T_hat_k = (1, 4/3, 1.2, 1) -> k = 2, whatever the
    # gradient statistics say (here they make DBW pick k = 1).
    T = [1.0, 1.5, 2.5, 4.0]
    k, obj = _choose_policy(4, 3.0, 0.1, -5.0, T, "blind")
    assert k == 2
    assert obj == [1.0 / 1.0, 2.0 / 1.5, 3.0 / 2.5, 4.0 / 4.0]
    assert _choose(4, 3.0, 0.1, -5.0, T)[0] == 1
    # all DBW gains negative (N = 0): DBW waits for all, B-DBW still maximises k / T
    assert _choose(4, 4.0, 0.0, 2.0, T)[0] == 4
    assert _choose_policy(4, 4.0, 0.0, 2.0, T, "blind")[0] == 2


def test_blind_ties_go_to_largest_k_and_rest_of_rule_holds():
    k, _ = _choose_policy(5, 1.0, 1.0, 1.0, [1.0, 2.0, 3.0, 4.0, 5.0], "blind")   # k / k = 1 for all k
    assert k == 5
    # before the first smoothness estimate: n
    k, obj = _choose_policy(5, 1.0, 1.0, 1.0, [1.0, 2.0, 3.0, 4.0, 5.0], "blind", hL=False)
    assert k == 5 and obj is None
    # the loss guard still applies
    T = [1.0, 1.5, 2.5, 4.0, 8.0]
    assert _choose_policy(5, 1.0, 1.0, 1.0, T, "blind", k_prev=3)[0] == 2
    assert _choose_policy(5, 1.0, 1.0, 1.0, T, "blind", F=(1.0, 1.02), k_prev=3)[0] == 4
    # missing estimates are not eligible
    assert _choose_policy(4, 1.0, 1.0, 1.0, [None, 1.5, None, 4.0], "blind")[0] == 2


def test_static_policy_overrides_the_choice_and_keeps_the_objective():
    T = [1.0, 1.5, 2.0, 2.5, 3.0, 3.5]
    k_dbw, obj_dbw = _choose(6, 3.0, 0.1, -5.0, T, F=(1.0, 1.02), k_prev=3)
    for ks in (1, 3, 6):
        k, obj = _choose_policy(6, 3.0, 0.1, -5.0, T, "static", k_static=ks, F=(1.0, 1.02), k_prev=3)
        assert k == ks and obj == obj_dbw
    k, obj = _choose_policy(6, 3.0, 0.1, -5.0, T, "static", k_static=2, hL=False)
    assert k == 2 and obj is None
    with pytest.raises(ValueError):
        _choose_policy(6, 3.0, 0.1, -5.0, T, "oracle")


def test_static_policy_trajectory_and_push_interrupt_rows():
    # A static run keeps k; under Push & Interrupt each iteration leaves
    # exactly k_t samples in row k_{t-1} (k_{-1} = n).
    cfg = _tiny_cfg(policy="static", k_static=2, clock="psi")
    X, y = gen.dataset(cfg)
    orc = dbw.DBWOracle(cfg, init_params(cfg))
    for t in range(5):
        Xt, yt = gather(X, y, gen.batch_indices(cfg, t))
        rec = orc.step(Xt, yt, gen.round_trip_ticks(cfg, t))
        assert rec["k"] == 2 and sum(rec["computed"]) == 2
    cnt = np.array(orc.cnt)
    assert cnt[cfg.n - 1].tolist() == [1, 1] + [0] * (cfg.n - 2)      # iteration 0, row n
    assert cnt[1].tolist() == [4, 4] + [0] * (cfg.n - 2)              # iterations 1-4, row 2
    assert cnt.sum() == 2 * 5
