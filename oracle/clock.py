"""Virtual clocks of the simulated cluster (Sect. 2 and Sect. 3.2).

Test infrastructure only (see the package docstring).

Both clocks turn the round-trip times tau_{i,t} of an iteration (integer
ticks, one per worker: the time worker i needs to fetch the parameters,
compute a gradient and send it) into arrival offsets o_i from the start s_t
of the iteration.  The PS uses the k_t smallest offsets; the next iteration
starts at s_{t+1} = s_t + (k_t-th smallest offset).

Fresh start: every worker starts computing w_t at s_t, so o_i = tau_{i,t},
and all n arrivals are samples of iteration t (late workers still report).

Push & Wait (the paper's PsW): the PS pushes w_{t+1} as soon as it holds
k_t gradients of w_t.  A worker still computing a gradient of an older
vector finishes it first and then takes the most recent vector of its queue.
With b_i the time worker i becomes free:
  * worker i computes w_t when it is idle at the push (b_i <= s_t) or becomes
    free before the next one (b_i < s_{t+1}); its gradient of w_t then
    arrives at max(s_t, b_i) + tau_{i,t}, the offset
    o_i = max(s_t, b_i) - s_t + tau_{i,t}, and b_i becomes s_t + o_i;
  * otherwise it is still busy at s_{t+1} and skips w_t: it sends no gradient
    of w_t (no sample) and b_i is unchanged.
A worker that skips w_t has o_i > s_{t+1} - s_t, so it is never among the
first k_t; the k_t-th smallest offset over all workers is therefore the one
over the workers that compute w_t.  A worker that becomes free exactly at
s_{t+1} takes w_{t+1}.  The samples of iteration t are the sorted offsets of
the workers that compute w_t (fewer than n when some skip: the censoring of
the estimator's data).

Push & Interrupt (the paper's PsI): the push of w_{t+1} interrupts every
worker, which drops the gradient it is computing and starts on w_{t+1}.
Every iteration therefore starts afresh, o_i = tau_{i,t}, but only the
workers that deliver before the push complete: the first k_t in (offset,
worker index) order.  Their offsets are the samples; the later n - k_t are
censored.
"""
from __future__ import annotations


class FreshClock:
    """Every worker starts each iteration afresh."""

    def __init__(self, n: int):
        self.n = n
        self.s = 0

    def offsets(self, tau):
        return [int(x) for x in tau]

    def advance(self, offsets, k: int):
        """End of the iteration after k arrivals; returns the sorted samples
        and, per worker, whether it computed this iteration's gradient."""
        srt = sorted(offsets)
        self.s += srt[k - 1]
        return srt, [True] * self.n


class PsWClock:
    """Push & Wait: late workers finish their current computation first."""

    def __init__(self, n: int):
        self.n = n
        self.s = 0
        self.busy = [0] * n       # time each worker becomes free

    def offsets(self, tau):
        return [max(self.s, b) - self.s + int(x) for b, x in zip(self.busy, tau)]

    def advance(self, offsets, k: int):
        s_next = self.s + sorted(offsets)[k - 1]
        computed = [b <= self.s or b < s_next for b in self.busy]
        samples = sorted(o for o, c in zip(offsets, computed) if c)
        self.busy = [self.s + o if c else b for b, o, c in zip(self.busy, offsets, computed)]
        self.s = s_next
        return samples, computed


class PsIClock:
    """Push & Interrupt: the push restarts every worker on the new vector."""

    def __init__(self, n: int):
        self.n = n
        self.s = 0

    def offsets(self, tau):
        return [int(x) for x in tau]

    def advance(self, offsets, k: int):
        order = sorted(range(self.n), key=lambda i: (offsets[i], i))
        done = order[:k]
        self.s += offsets[order[k - 1]]
        computed = [False] * self.n
        for i in done:
            computed[i] = True
        return [offsets[i] for i in done], computed


def make_clock(kind: str, n: int):
    if kind == "fresh":
        return FreshClock(n)
    if kind == "psw":
        return PsWClock(n)
    if kind == "psi":
        return PsIClock(n)
    raise ValueError(f"unknown clock {kind!r}")
