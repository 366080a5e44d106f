"""Pins of the oracle's virtual clocks (oracle/clock.py): the Push & Wait rule
of Sect. 2 against a hand-worked case and an independent event-driven
simulation of the cluster, its reduction to the fresh-start clock when the
PS always waits for every worker, and the invariants of the censoring."""
import heapq

import numpy as np
import pytest

from oracle.clock import FreshClock, PsIClock, PsWClock, make_clock


def test_psw_hand_worked_case():
    # n = 3.  Iteration 0: all idle at s0 = 0, tau = (2, 5, 9), k0 = 1 ->
    #   offsets (2, 5, 9), s1 = 2, all three compute w_0, busy = (2, 5, 9).
    # Iteration 1: tau = (3, 1, 1), k1 = 2 -> worker 0 idle: 3; worker 1
    #   free at 5: 5 - 2 + 1 = 4; worker 2 free at 9: 9 - 2 + 1 = 8.
    #   s2 = 2 + 4 = 6.  Worker 2 is still busy at 6 (9 >= 6): it skips w_1.
    #   Samples (3, 4); busy = (5, 6, 9).
    # Iteration 2: tau = (4, 4, 4), k2 = 3 -> worker 0 free at 5 <= 6: 4;
    #   worker 1 free at 6 <= 6: 4; worker 2 free at 9: 9 - 6 + 4 = 7.
    #   s3 = 6 + 7 = 13; 9 < 13 so worker 2 computes w_2.  Samples (4, 4, 7).
    c = PsWClock(3)
    o = c.offsets([2, 5, 9])
    assert o == [2, 5, 9]
    samples, computed = c.advance(o, 1)
    assert (samples, computed, c.s, c.busy) == ([2, 5, 9], [True] * 3, 2, [2, 5, 9])
    o = c.offsets([3, 1, 1])
    assert o == [3, 4, 8]
    samples, computed = c.advance(o, 2)
    assert (samples, computed, c.s, c.busy) == ([3, 4], [True, True, False], 6, [5, 6, 9])
    o = c.offsets([4, 4, 4])
    assert o == [4, 4, 7]
    samples, computed = c.advance(o, 3)
    assert (samples, computed, c.s, c.busy) == ([4, 4, 7], [True] * 3, 13, [10, 10, 13])


def _simulate(tau, ks):
    """Event-driven run of the cluster under Push & Wait: a heap of gradient
    completions in time order.  The PS counts the gradients of the current
    vector as they arrive (ties by worker index) and pushes w_{t+1} when the
    k_t-th gradient of w_t arrives.  After all completions of one instant
    are counted, every worker that completed at that instant takes the
    newest pushed vector it has not computed (a push at the same instant
    included), or waits idle for the next push.  Returns the push times and,
    per iteration, the sorted arrival offsets of the workers that computed
    it."""
    T, n = len(ks), len(tau[0])
    s = [0]
    heap = [(int(tau[0][i]), i, 0) for i in range(n)]
    heapq.heapify(heap)
    arrivals = [[] for _ in range(T)]
    got = 0
    idle = []
    while heap:
        f = heap[0][0]
        done = []
        while heap and heap[0][0] == f:
            _, i, it = heapq.heappop(heap)
            arrivals[it].append(f - s[it])
            done.append((i, it))
            if it == len(s) - 1 and len(s) <= T:
                got += 1
                if got == ks[it]:
                    s.append(f)     # push of w_{it+1}
                    got = 0
                    if len(s) - 1 < T:
                        for j in idle:
                            heapq.heappush(heap, (f + int(tau[len(s) - 1][j]), j, len(s) - 1))
                    idle = []
        latest = len(s) - 1
        for i, it in done:
            if latest < T and it < latest:
                heapq.heappush(heap, (f + int(tau[latest][i]), i, latest))
            elif latest < T:
                idle.append(i)
    return s, [sorted(a) for a in arrivals]


@pytest.mark.parametrize("seed", range(8))
def test_psw_matches_event_simulation(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 9))
    T = 25
    tau = rng.integers(1, 40, size=(T, n))
    if seed % 2:
        tau[:, 0] *= 6                      # one slow worker: it skips iterations
    ks = [int(rng.integers(1, n + 1)) for _ in range(T)]
    s_ref, arr_ref = _simulate(tau, ks)
    c = PsWClock(n)
    for t in range(T):
        o = c.offsets(tau[t])
        samples, computed = c.advance(o, ks[t])
        assert c.s == s_ref[t + 1], t
        assert samples == arr_ref[t], t
        assert sum(computed) == len(samples) >= ks[t]


def test_psw_equals_fresh_start_when_waiting_for_all():
    # With k_t = n the PS waits for every worker, so nobody is busy at a push.
    rng = np.random.default_rng(3)
    n = 6
    a, b = PsWClock(n), FreshClock(n)
    for _ in range(30):
        tau = rng.integers(1, 100, size=n)
        oa, ob = a.offsets(tau), b.offsets(tau)
        assert oa == ob
        assert a.advance(oa, n) == b.advance(ob, n)
        assert a.s == b.s


def test_psw_censoring_invariants():
    rng = np.random.default_rng(4)
    n = 8
    c = make_clock("psw", n)
    for t in range(200):
        tau = rng.integers(1, 50, size=n)
        tau[3] *= 20                         # a straggler
        o = c.offsets(tau)
        assert all(x >= y for x, y in zip(o, tau))         # never earlier than its own round trip
        k = int(rng.integers(1, n + 1))
        s0 = c.s
        busy0 = list(c.busy)
        samples, computed = c.advance(o, k)
        assert c.s - s0 == sorted(o)[k - 1]
        assert len(samples) == sum(computed) >= k
        for i in range(n):
            if not computed[i]:
                assert busy0[i] >= c.s and c.busy[i] == busy0[i]    # still busy at the push: skipped
                assert o[i] > c.s - s0
            else:
                assert c.busy[i] == s0 + o[i]
    with pytest.raises(ValueError):
        make_clock("sundial", 2)


def test_psi_hand_worked_case():
    # n = 3, tau = (2, 5, 9), k = 2: workers 0 and 1 deliver at 2 and 5, the
    # push at 5 interrupts worker 2.  Then tau = (4, 4, 4), k = 2: ties by
    # index, worker 2 is interrupted at the push at 5 + 4 = 9.
    c = make_clock("psi", 3)
    o = c.offsets([2, 5, 9])
    assert o == [2, 5, 9]
    assert c.advance(o, 2) == ([2, 5], [True, True, False]) and c.s == 5
    o = c.offsets([4, 4, 4])
    assert c.advance(o, 2) == ([4, 4], [True, True, False]) and c.s == 9
    o = c.offsets([7, 1, 3])
    assert c.advance(o, 1) == ([1], [False, True, False]) and c.s == 10


@pytest.mark.parametrize("seed", range(4))
def test_psi_is_fresh_start_censored_at_k(seed):
    # Every push restarts all workers, so the timing is the fresh-start one;
    # only the first k_t arrivals (by offset, then index, as the PS selects)
    # complete.
    from oracle.ps import select_fastest
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(2, 12))
    a, b = PsIClock(n), FreshClock(n)
    for _ in range(40):
        tau = rng.integers(1, 30, size=n)           # small range: many ties
        k = int(rng.integers(1, n + 1))
        oa, ob = a.offsets(tau), b.offsets(tau)
        assert oa == ob
        samples, computed = a.advance(oa, k)
        fresh, _ = b.advance(ob, k)
        assert samples == fresh[:k] and a.s == b.s
        _, mask = select_fastest(oa, k)
        assert computed == [bool(m) for m in mask]
