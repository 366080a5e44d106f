"""Seeded synthetic inputs for the DBW simulation.

Every random number the simulation consumes is drawn here and handed to both
the CPU oracle and the GPU path as plain arrays: the finite dataset, the
initial parameters, the per-iteration minibatch row indices of every worker
and the per-iteration round-trip ticks of every worker.

Seeding: workload c uses ``SeedSequence(cfg.seed)`` with five independent
streams (features, labels, init, minibatch indices, times).  Per-iteration
draws use ``spawn_key=(stream, t)`` so that iteration t can be regenerated
without replaying iterations 0..t-1.
"""
from __future__ import annotations

import functools

import numpy as np

from .configs import CNN, MLP, SOFTMAX, TICKS_PER_UNIT, DBWConfig

STREAM_FEATURES, STREAM_LABELS, STREAM_INIT, STREAM_INDICES, STREAM_TIMES = range(5)


def _rng(cfg: DBWConfig, stream: int, t: int | None = None) -> np.random.Generator:
    key = (stream,) if t is None else (stream, int(t))
    return np.random.default_rng(np.random.SeedSequence(cfg.seed, spawn_key=key))


@functools.lru_cache(maxsize=4)
def dataset(cfg: DBWConfig) -> tuple[np.ndarray, np.ndarray]:
    """The finite dataset: features float32 [S][d], labels int32 [S]."""
    rf = _rng(cfg, STREAM_FEATURES)
    if cfg.features == "uniform":
        X = rf.random((cfg.S, cfg.d), dtype=np.float32)
    elif cfg.features == "normal":
        X = rf.standard_normal((cfg.S, cfg.d), dtype=np.float32)
    else:
        raise ValueError(f"unknown feature law {cfg.features!r}")
    if cfg.sparsity > 0.0:
        X[rf.random((cfg.S, cfg.d), dtype=np.float32) < cfg.sparsity] = 0.0
    rl = _rng(cfg, STREAM_LABELS)
    if cfg.labels == "uniform":
        y = rl.integers(0, cfg.C, size=cfg.S, dtype=np.int32)
    elif cfg.labels == "teacher":
        # Labels of a random linear teacher: the gradient norm dominates the
        # minibatch variance early in training.
        Wt = rl.standard_normal((cfg.d, cfg.C)).astype(np.float32)
        y = np.argmax(X @ Wt, axis=1).astype(np.int32)
    else:
        raise ValueError(f"unknown label law {cfg.labels!r}")
    X.setflags(write=False)
    y.setflags(write=False)
    return X, y


def init_params(cfg: DBWConfig) -> np.ndarray:
    """Initial parameter vector w_0, float32 [P]."""
    r = _rng(cfg, STREAM_INIT)
    if cfg.model == SOFTMAX:
        return r.normal(0.0, cfg.init_std, size=(cfg.d, cfg.C)).astype(np.float32).ravel()
    if cfg.model == MLP:
        # Kaiming-normal (fan_in, gain sqrt 2) weights, zero biases.
        W1 = r.normal(0.0, np.sqrt(2.0 / cfg.d), size=(cfg.d, cfg.H)).astype(np.float32)
        W2 = r.normal(0.0, np.sqrt(2.0 / cfg.H), size=(cfg.H, cfg.C)).astype(np.float32)
        return np.concatenate([W1.ravel(), np.zeros(cfg.H, np.float32),
                               W2.ravel(), np.zeros(cfg.C, np.float32)])
    if cfg.model == CNN:
        # PyTorch's default for convolution and linear layers: weights and
        # biases uniform in +-1/sqrt(fan_in)
        parts = []
        # layout: the fully connected layers first, then the convolutions
        for shape, fan_in in (((800, cfg.H), 800), ((cfg.H,), 800), ((cfg.H, cfg.C), cfg.H), ((cfg.C,), cfg.H),
                              ((20, 1, 5, 5), 25), ((20,), 25), ((50, 20, 5, 5), 500), ((50,), 500)):
            bound = 1.0 / np.sqrt(fan_in)
            parts.append(r.uniform(-bound, bound, size=shape).astype(np.float32).ravel())
        return np.concatenate(parts)
    raise ValueError(cfg.model)


def batch_indices(cfg: DBWConfig, t: int) -> np.ndarray:
    """Row indices of worker i's minibatch at iteration t, int32 [n][B].
    Each worker samples B rows of the whole dataset uniformly with
    replacement, independently of the other workers."""
    return _rng(cfg, STREAM_INDICES, t).integers(0, cfg.S, size=(cfg.n, cfg.B), dtype=np.int32)


def round_trip_times(cfg: DBWConfig, t: int) -> np.ndarray:
    """tau_{i,t} in time units, float64 [n]."""
    tm = cfg.times
    r = _rng(cfg, STREAM_TIMES, t)
    n = cfg.n
    if tm.kind == "shifted_exp":
        tau = tm.shift + r.exponential(1.0 / tm.rate, size=n)
    elif tm.kind == "pareto":
        u = r.random(n)
        tau = tm.scale * (1.0 - u) ** (-1.0 / tm.shape)
    elif tm.kind == "uniform":
        tau = tm.low + (tm.high - tm.low) * r.random(n)
    else:
        raise ValueError(f"unknown time law {tm.kind!r}")
    if tm.slow_workers:
        tau[list(tm.slow_workers)] *= tm.slow_factor
    if tm.straggler_prob > 0.0:
        hit = r.random(n) < tm.straggler_prob
        tau[hit] *= tm.straggler_factor
    return tau


def round_trip_ticks(cfg: DBWConfig, t: int) -> np.ndarray:
    """tau_{i,t} rounded to integer ticks of 2**-20 units (>= 1), int64 [n]."""
    ticks = np.rint(round_trip_times(cfg, t) * TICKS_PER_UNIT).astype(np.int64)
    return np.maximum(ticks, 1)


def gather(X: np.ndarray, y: np.ndarray, idx: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Materialise the minibatches: X_t float32 [n][B][d], y_t int32 [n][B]."""
    return X[idx], y[idx]


def iteration_inputs(cfg: DBWConfig, t: int):
    """(X_t, y_t, ticks_t) for iteration t."""
    X, y = dataset(cfg)
    Xt, yt = gather(X, y, batch_indices(cfg, t))
    return Xt, yt, round_trip_ticks(cfg, t)
