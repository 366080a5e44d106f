"""The DBW controller and the full iteration, float64 (Sect. 3).

Choice of k_t at the start of iteration t (Sect. 3.3):
  * D-window means of past end-of-iteration estimates (Eqs. varianceoverD,
    normsquareoverD, LoverD): the mean of the most recent min(D, available)
    entries.
  * gain (Eq. gain):  G_k = (eta - L eta^2/2) N - (L eta^2/2) V / k,  k = 1..n
  * greedy choice (Eq. greedy): k* = argmax_k G_k / T_hat_k; k* = n when every
    G_k < 0; exact ties go to the largest k (the cautious side).
  * loss guard (Eq. greedy2): if F_hat_{t-1} > beta F_hat_{t-2} and
    k_{t-1} < n then k_t = max(k*, k_{t-1} + 1).
  * Before any L estimate exists (t = 0, 1) k_t = n; k_{-1} is taken as n.

Variants the paper compares (Sect. 4): a static k (k_t = k_static at every
iteration; the objective is still reported), and B-DBW, which takes the gain
G_k = k (the number of aggregated gradients) and keeps the rest of the rule.
The time estimate is the constrained one (Eq. quadratic_opt) or the naive
mean of cell (k, k) (Sect. 3.2).

End of iteration t (Sect. 3.1, Sect. 3.2):
  * push V+_t, N+_t, F_hat_t;
  * for t >= 1, L+_t = 2 (eta N+_{t-1} - (F_hat_{t-1} - F_hat_t))
                     / (eta^2 (N+_{t-1} + V+_{t-1} / k_{t-1}))      (Eq. estimateL)
    is pushed when the denominator is positive;
  * the arrival offsets of iteration t (from the round-trip ticks, through the
    clock of the configuration: fresh start or Push & Wait, oracle/clock.py)
    of the workers that computed w_t are recorded, in arrival order, as
    samples of row h = k_{t-1} (late workers still notify completion);
  * the virtual clock advances by the k_t-th smallest offset.

Test infrastructure only (see the package docstring).
"""
from __future__ import annotations

import numpy as np

from . import model, ps
from .clock import make_clock
from .time_estimator import naive_estimate, time_estimate


def window_mean(hist, D: int):
    """Mean of the last min(D, len(hist)) entries; None if hist is empty."""
    if not hist:
        return None
    last = hist[-D:]
    return sum(last) / len(last)


def gains(V: float, N: float, L: float, eta: float, n: int):
    """G_k for k = 1..n (Eq. gain), as a list indexed k-1."""
    a = eta - L * eta * eta / 2.0
    b = L * eta * eta / 2.0
    return [a * N - b * V / k for k in range(1, n + 1)]


def choose_k(n: int, eta: float, beta: float, D: int, hV, hN, hL, F_hist, k_prev: int,
             T_hat, policy: str = "dbw", k_static: int = 0):
    """Returns (k_t, objective) with objective[k-1] = G_k / T_hat_k (None
    before the first L estimate).  k whose T_hat_k is missing is not eligible.
    policy "blind" (B-DBW) uses G_k = k; "static" returns k_static."""
    if policy not in ("dbw", "static", "blind"):
        raise ValueError(f"unknown policy {policy!r}")
    if not hL:
        k_star, objective = n, None
    else:
        if policy == "blind":
            G = [float(k) for k in range(1, n + 1)]
        else:
            V = window_mean(hV, D)
            N = window_mean(hN, D)
            L = window_mean(hL, D)
            G = gains(V, N, L, eta, n)
        objective = [(G[k - 1] / T_hat[k - 1]) if (T_hat[k - 1] is not None and T_hat[k - 1] > 0)
                     else None for k in range(1, n + 1)]
        eligible = [k for k in range(1, n + 1) if objective[k - 1] is not None]
        if not eligible or max(G) < 0.0:
            k_star = n
        else:
            best = max(objective[k - 1] for k in eligible)
            k_star = max(k for k in eligible if objective[k - 1] == best)
    k_t = k_star
    if len(F_hist) >= 2 and F_hist[-1] > beta * F_hist[-2] and k_prev < n:
        k_t = max(k_star, k_prev + 1)
    if policy == "static":
        k_t = k_static
    return k_t, objective


def l_estimate(eta: float, N_prev: float, V_prev: float, k_prev: int, F_prev: float,
               F_now: float):
    """L+_t from the previous iteration's estimates (Eq. estimateL); None when
    the denominator is not positive."""
    den = eta * eta * (N_prev + V_prev / k_prev)
    if not den > 0.0:
        return None
    return 2.0 * (eta * N_prev - (F_prev - F_now)) / den


class DBWOracle:
    """State and one-iteration step of the DBW parameter server."""

    def __init__(self, cfg, w0):
        self.cfg = cfg
        n = cfg.n
        self.w = np.asarray(w0, dtype=np.float64).copy()
        self.hV, self.hN, self.hL, self.F = [], [], [], []
        self.ks = []               # k_0, k_1, ...
        self.k_prev = n            # k_{-1}
        self.t = 0
        self.cnt = [[0] * n for _ in range(n)]
        self.tsum = [[0] * n for _ in range(n)]
        self.vclock = make_clock(getattr(cfg, "clock", "fresh"), n)
        self.clock = 0

    # -- pieces ------------------------------------------------------------
    def time_estimate(self):
        if getattr(self.cfg, "estimator", "isotonic") == "naive":
            return naive_estimate(self.cnt, self.tsum)
        if not any(any(r) for r in self.cnt):
            return [None] * self.cfg.n
        return time_estimate(self.cnt, self.tsum)

    def choose(self, T_hat):
        c = self.cfg
        return choose_k(c.n, c.eta, c.beta, c.D, self.hV, self.hN, self.hL, self.F,
                        self.k_prev, T_hat, policy=getattr(c, "policy", "dbw"),
                        k_static=getattr(c, "k_static", 0))

    def record_times(self, offsets, k_t):
        """Bookkeeping of the arrival offsets of this iteration (row k_{t-1}):
        the samples of the workers that computed w_t, and the clock."""
        samples, computed = self.vclock.advance(offsets, k_t)
        h = self.k_prev
        for i, v in enumerate(samples):
            self.cnt[h - 1][i] += 1
            self.tsum[h - 1][i] += v
        self.clock = self.vclock.s
        return computed

    # -- the iteration -------------------------------------------------------
    def step(self, Xt, yt, ticks, T_hat=None, k_force=None):
        """One DBW iteration on minibatches Xt [n][B][d], yt [n][B] and
        round-trip ticks [n].  ``T_hat`` overrides the time estimate and
        ``k_force`` the choice (static-k runs, lockstep tests)."""
        c = self.cfg
        offsets = self.vclock.offsets(ticks)
        if T_hat is None:
            T_hat = self.time_estimate()
        k_t, objective = self.choose(T_hat)
        if k_force is not None:
            k_t = int(k_force)
        V_window = window_mean(self.hV, c.D)
        G, loss = model.worker_grads(c, self.w, Xt, yt)
        sel, mask = ps.select_fastest(offsets, k_t)
        g = ps.aggregate(G, sel)
        st = ps.grad_stats(G, sel, g, loss, V_window if V_window is not None else 0.0)
        w_next = ps.sgd_update(self.w, g, c.eta)
        # bookkeeping
        L_new = None
        if self.t >= 1:
            L_new = l_estimate(c.eta, self.hN[-1], self.hV[-1], self.k_prev, self.F[-1],
                               st["F_hat"])
        self.hV.append(st["V_plus"])
        self.hN.append(st["N_plus"])
        self.F.append(st["F_hat"])
        if L_new is not None:
            self.hL.append(L_new)
        computed = self.record_times(offsets, k_t)
        rec = {"t": self.t, "k": k_t, "b": c.n - k_t, "objective": objective,
               "offsets": offsets, "computed": computed,
               "T_hat": T_hat, "G": G, "loss": loss, "sel": sel, "mask": mask, "g": g,
               "w_prev": self.w, "w": w_next, "L_plus": L_new, **st}
        self.w = w_next
        self.ks.append(k_t)
        self.k_prev = k_t
        self.t += 1
        return rec

    def export_state(self):
        """The estimator state a GPU context needs to continue from here."""
        D = self.cfg.D
        return {
            "t": self.t, "k_prev": self.k_prev,
            "hV": list(self.hV[-D:]), "hN": list(self.hN[-D:]), "hL": list(self.hL[-D:]),
            "F_prev": self.F[-1] if len(self.F) >= 1 else 0.0,
            "F_prev2": self.F[-2] if len(self.F) >= 2 else 0.0,
            "nF": min(len(self.F), 2),
            "V_last": self.hV[-1] if self.hV else 0.0,
            "N_last": self.hN[-1] if self.hN else 0.0,
            "cnt": [list(r) for r in self.cnt], "tsum": [list(r) for r in self.tsum],
            "clock": self.clock,
        }
