"""Pins of the oracle's order-statistic time estimator (Sect. 3.2,
Eq. quadratic_opt): hand-solved cases, reductions to 1-D isotonic regression
(scipy) and to empirical means, the max-min formula of isotonic regression by
brute force on tiny grids, an independent numerical QP solve, and long-run
closed forms of expected order statistics."""
import json
import math
import os
from fractions import Fraction
from itertools import combinations

import numpy as np
import pytest
from scipy.optimize import isotonic_regression, minimize

from dbw_inputs import TICKS_PER_UNIT, DBWConfig, TimeModel
from dbw_inputs import generate as gen
from oracle import time_estimator as te

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "time_estimate_cases.json")


def _full_grid_leq(n):
    """leq[(h',k')][(h,k)]: x_{h',k'} <= x_{h,k} is implied by the three
    constraint families written literally on the full n x n grid."""
    cells = [(h, k) for h in range(1, n + 1) for k in range(1, n + 1)]
    succ = {c: [] for c in cells}
    for h in range(1, n + 1):
        for k in range(1, n):
            succ[(h, k)].append((h, k + 1))            # x_{h,k} <= x_{h,k+1}
    for h in range(1, n):
        for k in range(1, n + 1):
            succ[(h + 1, k)].append((h, k))            # x_{h+1,k} <= x_{h,k}
    for k in range(1, n):
        succ[(k, k)].append((k + 1, k + 1))            # x_{k,k} <= x_{k+1,k+1}
    reach = {}
    for c in cells:
        seen, stack = {c}, [c]
        while stack:
            u = stack.pop()
            for v in succ[u]:
                if v not in seen:
                    seen.add(v)
                    stack.append(v)
        reach[c] = seen
    return reach


def _random_grid(rng, n, p_row=0.5, full_rows=True, max_cnt=4, scale=50):
    cnt = [[0] * n for _ in range(n)]
    tsum = [[0] * n for _ in range(n)]
    rows = [h for h in range(n) if rng.random() < p_row] or [int(rng.integers(0, n))]
    for h in rows:
        for k in range(n):
            if full_rows or rng.random() < 0.6:
                c = int(rng.integers(1, max_cnt + 1))
                cnt[h][k] = c
                tsum[h][k] = int(sum(rng.integers(1, scale, size=c)))
    return cnt, tsum


def test_golden_hand_solved_cases():
    with open(GOLDEN) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        got = te.time_estimate(case["cnt"], case["tsum"], exact=True)
        assert got == [Fraction(x) for x in case["T_hat"]], case["name"]


def test_single_row_is_one_dimensional_isotonic_regression():
    # With one sampled row every induced constraint is along the row, so the
    # fit is 1-D weighted isotonic regression (scipy's PAVA).
    rng = np.random.default_rng(31)
    for _ in range(40):
        n = int(rng.integers(2, 12))
        h = int(rng.integers(1, n + 1))
        cnt = [[0] * n for _ in range(n)]
        tsum = [[0] * n for _ in range(n)]
        for k in range(n):
            cnt[h - 1][k] = int(rng.integers(1, 5))
            tsum[h - 1][k] = int(rng.integers(1, 100)) * cnt[h - 1][k]
        fit = te.fit_observed(cnt, tsum)
        y = np.array([tsum[h - 1][k] / cnt[h - 1][k] for k in range(n)])
        w = np.array([cnt[h - 1][k] for k in range(n)], dtype=float)
        ref = isotonic_regression(y, weights=w, increasing=True).x
        got = np.array([float(fit[(h, k)]) for k in range(1, n + 1)])
        np.testing.assert_allclose(got, ref, rtol=1e-12)
        # T_hat_k = fitted (h, min(k, h)), the largest sampled value below (k,k)
        T = te.time_estimate(cnt, tsum)
        for k in range(1, n + 1):
            assert T[k - 1] == pytest.approx(got[min(k, h) - 1], rel=1e-12)


def test_consistent_data_returns_empirical_means():
    # x_{h,k} = 10 k - h satisfies all three families; sampled means equal to
    # it are already optimal (Sect. 3.2: without binding constraints the
    # estimate is the empirical average).
    rng = np.random.default_rng(32)
    for _ in range(20):
        n = int(rng.integers(2, 9))
        cnt, _ = _random_grid(rng, n, full_rows=False)
        tsum = [[cnt[h][k] * (10 * (k + 1) - (h + 1)) for k in range(n)] for h in range(n)]
        fit = te.fit_observed(cnt, tsum)
        emp = te.empirical_means(cnt, tsum)
        for (h, k), x in fit.items():
            assert x == emp[h - 1][k - 1]


def test_contracted_order_equals_full_grid_order():
    rng = np.random.default_rng(33)
    for _ in range(60):
        n = int(rng.integers(1, 8))
        cnt, _ = _random_grid(rng, n)
        nodes, edges = te.order_graph(cnt)
        succ = {i: [] for i in range(len(nodes))}
        for u, v in edges:
            succ[u].append(v)
        full = _full_grid_leq(n)
        for i, a in enumerate(nodes):
            seen, stack = {i}, [i]
            while stack:
                u = stack.pop()
                for v in succ[u]:
                    if v not in seen:
                        seen.add(v)
                        stack.append(v)
            got = {nodes[j] for j in seen}
            want = {b for b in nodes if b in full[a]}
            assert got == want, (n, a)


def _maxmin_brute_force(obs, leq, c, s):
    """Isotonic regression by the max-min formula: x_v = max over upper sets
    U containing v of min over lower sets L containing v of the weighted mean
    of U & L (Robertson, Wright & Dykstra 1988, Thm 1.4.4)."""
    m = len(obs)
    ups, lows = [], []
    for r in range(1, m + 1):
        for sub in combinations(range(m), r):
            S = set(sub)
            if all(b in S for a in S for b in range(m) if leq[a][b]):
                ups.append(S)
            if all(b in S for a in S for b in range(m) if leq[b][a]):
                lows.append(S)
    out = []
    for v in range(m):
        best = None
        for U in ups:
            if v not in U:
                continue
            worst = None
            for Lw in lows:
                if v not in Lw:
                    continue
                I = U & Lw
                val = Fraction(sum(s[i] for i in I), sum(c[i] for i in I))
                worst = val if worst is None or val < worst else worst
            best = worst if best is None or worst > best else best
        out.append(best)
    return out


def test_tiny_grids_match_max_min_brute_force():
    rng = np.random.default_rng(34)
    checked = 0
    while checked < 60:
        n = int(rng.integers(1, 4))
        cnt, tsum = _random_grid(rng, n, full_rows=False, scale=30)
        obs = [(h + 1, k + 1) for h in range(n) for k in range(n) if cnt[h][k] > 0]
        if len(obs) > 7:
            continue
        full = _full_grid_leq(n)
        leq = [[b in full[a] for b in obs] for a in obs]
        c = [cnt[h - 1][k - 1] for h, k in obs]
        s = [tsum[h - 1][k - 1] for h, k in obs]
        ref = _maxmin_brute_force(obs, leq, c, s)
        fit = te.fit_observed(cnt, tsum)
        assert [fit[o] for o in obs] == ref
        checked += 1


def test_moderate_grids_match_numerical_qp():
    # Independent numerical solve (SLSQP) of Eq. quadratic_opt over the
    # sampled cells with every pairwise order relation as a constraint.
    rng = np.random.default_rng(35)
    for _ in range(6):
        n = int(rng.integers(4, 7))
        cnt, tsum = _random_grid(rng, n, p_row=0.4, scale=40)
        obs = [(h + 1, k + 1) for h in range(n) for k in range(n) if cnt[h][k] > 0]
        full = _full_grid_leq(n)
        c = np.array([cnt[h - 1][k - 1] for h, k in obs], float)
        m = np.array([tsum[h - 1][k - 1] / cnt[h - 1][k - 1] for h, k in obs])
        pairs = [(i, j) for i, a in enumerate(obs) for j, b in enumerate(obs)
                 if i != j and b in full[a]]
        A = np.zeros((len(pairs), len(obs)))
        for r, (i, j) in enumerate(pairs):
            A[r, i], A[r, j] = -1.0, 1.0        # x_j - x_i >= 0
        scale = float(np.max(m))
        ms, cs = m / scale, c / c.sum()
        x0 = np.full(len(obs), float(cs @ ms))       # a constant vector is feasible
        res = minimize(lambda x: float(cs @ (x - ms) ** 2), x0,
                       jac=lambda x: 2 * cs * (x - ms), method="SLSQP",
                       constraints=[{"type": "ineq", "fun": lambda x: A @ x, "jac": lambda x: A}],
                       options={"ftol": 1e-15, "maxiter": 5000})
        assert res.success
        fit = te.fit_observed(cnt, tsum)
        got = np.array([float(fit[o]) for o in obs])
        np.testing.assert_allclose(got / scale, res.x, rtol=0, atol=1e-6)


def _expected_order_stat_shifted_exp(n, k, shift, rate):
    return shift + sum(1.0 / j for j in range(n - k + 1, n + 1)) / rate


def _expected_order_stat_pareto(n, k, xm, alpha):
    lg = math.lgamma
    return xm * math.exp(lg(n + 1) + lg(n - k + 1 - 1 / alpha) - lg(n - k + 1) - lg(n + 1 - 1 / alpha))


@pytest.mark.parametrize("law", ["shifted_exp", "pareto"])
def test_long_run_matches_expected_order_statistics(law):
    # Waiting always for all n workers samples only row h = n, so T_hat_k is
    # the running mean of the k-th smallest tick, which converges to the
    # expected k-th order statistic of the round-trip law.
    n, iters = 5, 6000
    tm = (TimeModel(kind="shifted_exp", shift=1.0, rate=0.5) if law == "shifted_exp"
          else TimeModel(kind="pareto", scale=1.0, shape=4.5))
    cfg = DBWConfig(name="t", model="softmax", n=n, B=1, d=1, C=2, times=tm, seed=99)
    cnt = [[0] * n for _ in range(n)]
    tsum = [[0] * n for _ in range(n)]
    samples = [[] for _ in range(n)]
    for t in range(iters):
        srt = np.sort(gen.round_trip_ticks(cfg, t))
        for i in range(n):
            cnt[n - 1][i] += 1
            tsum[n - 1][i] += int(srt[i])
            samples[i].append(srt[i] / TICKS_PER_UNIT)
    T = te.time_estimate(cnt, tsum)
    for k in range(1, n + 1):
        expect = (_expected_order_stat_shifted_exp(n, k, 1.0, 0.5) if law == "shifted_exp"
                  else _expected_order_stat_pareto(n, k, 1.0, 4.5))
        se = np.std(samples[k - 1], ddof=1) / np.sqrt(iters)
        assert abs(T[k - 1] / TICKS_PER_UNIT - expect) < 5 * se + 1e-6, (k, expect)


def test_solution_is_feasible_and_blockwise_mean():
    rng = np.random.default_rng(36)
    for _ in range(20):
        n = int(rng.integers(3, 9))
        cnt, tsum = _random_grid(rng, n, p_row=0.5)
        fit = te.fit_observed(cnt, tsum)
        full = _full_grid_leq(n)
        for a, xa in fit.items():
            for b, xb in fit.items():
                if b in full[a]:
                    assert xa <= xb
        # every level set takes the weighted mean of its data
        levels = {}
        for (h, k), x in fit.items():
            levels.setdefault(x, []).append((h, k))
        for x, cells in levels.items():
            tot_c = sum(cnt[h - 1][k - 1] for h, k in cells)
            tot_s = sum(tsum[h - 1][k - 1] for h, k in cells)
            assert Fraction(tot_s, tot_c) == x


def test_naive_estimate_hand_worked_case():
    # n = 3.  Row 1: counts (2, 2, 2), sums (2, 6, 10) -> means (1, 3, 5).
    # Row 3: counts (1, 1, 1), sums (4, 5, 6).  The naive estimate reads the
    # diagonal: T_1 = cell (1,1) = 1, T_2 = cell (2,2) (empty) -> None,
    # T_3 = cell (3,3) = 6.  The constrained estimate pools the violated
    # diagonal relation x_{1,1} <= ... and has a value for every k.
    cnt = [[2, 2, 2], [0, 0, 0], [1, 1, 1]]
    tsum = [[2, 6, 10], [0, 0, 0], [4, 5, 6]]
    assert te.naive_estimate(cnt, tsum) == [1.0, None, 6.0]
    iso = te.time_estimate(cnt, tsum)
    assert None not in iso
    # quotients are rounded once: 1/3 of a tick is the double nearest 1/3
    assert te.naive_estimate([[3]], [[1]]) == [1 / 3]
    assert te.naive_estimate([[3]], [[2 ** 52 + 1]]) == [float(Fraction(2 ** 52 + 1, 3))]


def test_naive_estimate_equals_constrained_one_on_consistent_full_grids():
    # With every row sampled and means x_{h,k} = 10 k - h (every constraint
    # slack) the fit is the empirical mean, and T_hat_k is the fit at (k,k).
    rng = np.random.default_rng(33)
    for _ in range(10):
        n = int(rng.integers(2, 8))
        cnt = [[int(rng.integers(1, 4)) for _ in range(n)] for _ in range(n)]
        tsum = [[cnt[h][k] * (10 * (k + 1) - (h + 1)) for k in range(n)] for h in range(n)]
        assert te.naive_estimate(cnt, tsum) == te.time_estimate(cnt, tsum) == \
            [float(10 * k - k) for k in range(1, n + 1)]
