"""Workload descriptions for the DBW parameter-server simulation.

Each workload fixes the model shape (softmax regression or the 784-512-10
MLP), the number of logical workers n, the per-worker minibatch B, the
synthetic feature / label / init distributions and the round-trip-time law
of the virtual clock.  The five named workloads below are shaped like the
paper's experiments (28x28 or 32x32x3 inputs, 10 or 100 classes, Sect. 4);
every value is synthetic and seeded.

This module holds no arithmetic of the method itself: it only describes
inputs.  Both the CPU oracle and the GPU path read it.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Optional, Tuple

SOFTMAX = "softmax"
MLP = "mlp"
CNN = "cnn"     # 28x28 images: conv 5x5 (20) - pool - conv 5x5 (50) - pool - FC H - FC C

# Round trip times are kept as integer ticks of 2**-20 time units, so that
# sums of samples and their order are exact on every side.
TICKS_PER_UNIT = 1 << 20


@dataclass(frozen=True)
class TimeModel:
    """Law of the round-trip time tau_{i,t} of worker i at iteration t.

    kind = "shifted_exp": tau = shift + Exp(rate)
    kind = "pareto":      tau = scale * (1 - U) ** (-1 / shape)
    kind = "uniform":     tau = low + (high - low) * U
    Then: workers listed in ``slow_workers`` are ``slow_factor`` times slower
    in every iteration, and every (i, t) is independently ``straggler_factor``
    times slower with probability ``straggler_prob``.  The factor multiplies
    the whole tau, shift included.
    """

    kind: str = "shifted_exp"
    shift: float = 1.0
    rate: float = 1.0
    scale: float = 1.0
    shape: float = 2.5
    low: float = 0.0
    high: float = 1.0
    slow_workers: Tuple[int, ...] = ()
    slow_factor: float = 1.0
    straggler_prob: float = 0.0
    straggler_factor: float = 1.0


@dataclass(frozen=True)
class DBWConfig:
    name: str
    model: str            # SOFTMAX or MLP
    n: int                # logical workers
    B: int                # minibatch per worker
    d: int                # input features
    C: int                # classes
    H: int = 0            # hidden width (MLP only)
    S: int = 60000        # rows of the finite synthetic dataset
    iters: int = 50
    eta: float = 0.1      # learning rate, constant for every k
    D: int = 5            # window of past estimates averaged by DBW
    beta: float = 1.01    # loss-increase guard factor
    features: str = "uniform"   # "uniform" in [0,1) or "normal" N(0,1)
    sparsity: float = 0.0       # probability an entry is zeroed
    init_std: float = 0.01      # softmax W ~ N(0, init_std^2)
    times: TimeModel = field(default_factory=TimeModel)
    seed: int = 14696           # base of the seed sequence
    labels: str = "uniform"     # "uniform" or "teacher" (test fixture)
    clock: str = "fresh"        # "fresh": every worker starts each iteration afresh;
                                # "psw": Push & Wait, late workers finish their current gradient first;
                                # "psi": Push & Interrupt, late workers drop it (only k_t samples)
    policy: str = "dbw"         # choice of k: "dbw", "static" (k_static), "blind" (B-DBW)
    k_static: int = 0           # k of the static policy
    estimator: str = "isotonic" # time estimate: "isotonic" or "naive" (mean of cell (k,k))
    g_rows: str = "all"         # worker-gradient rows a GPU step writes: "all", "selected", "none"

    @property
    def param_count(self) -> int:
        """P: softmax W is [d][C] (no bias); the MLP is flattened as
        [W1 (d x H) | b1 (H) | W2 (H x C) | b2 (C)]."""
        if self.model == SOFTMAX:
            return self.d * self.C
        if self.model == CNN:
            return 20 * 25 + 20 + 50 * 20 * 25 + 50 + 800 * self.H + self.H + self.H * self.C + self.C
        return self.d * self.H + self.H + self.H * self.C + self.C

    def replace(self, **kw) -> "DBWConfig":
        return dataclasses.replace(self, **kw)


# The five workloads.  Seeds: SeedSequence(14696 + c) for workload c = 1..5.
C1 = DBWConfig(
    name="C1", model=SOFTMAX, n=4, B=32, d=784, C=10, S=60000, iters=50,
    features="uniform", sparsity=0.8, seed=14696 + 1,
    times=TimeModel(kind="shifted_exp", shift=1.0, rate=1.0),
)
C2 = DBWConfig(
    name="C2", model=SOFTMAX, n=16, B=128, d=784, C=10, S=60000, iters=200,
    features="uniform", seed=14696 + 2,
    times=TimeModel(kind="shifted_exp", shift=1.0, rate=0.5,
                    slow_workers=(0, 1), slow_factor=5.0),
)
C3 = DBWConfig(
    name="C3", model=SOFTMAX, n=64, B=256, d=3072, C=10, S=50000, iters=200,
    features="normal", seed=14696 + 3,
    times=TimeModel(kind="pareto", scale=1.0, shape=2.5),
)
C4 = DBWConfig(
    name="C4", model=MLP, n=32, B=64, d=784, C=10, H=512, S=60000, iters=100,
    features="uniform", seed=14696 + 4,
    times=TimeModel(kind="shifted_exp", shift=1.0, rate=1.0),
)
C5 = DBWConfig(
    name="C5", model=SOFTMAX, n=256, B=512, d=3072, C=100, S=50000, iters=50,
    features="normal", seed=14696 + 5,
    times=TimeModel(kind="shifted_exp", shift=1.0, rate=0.2,
                    straggler_prob=0.1, straggler_factor=10.0),
)

# The paper's MNIST network shape (two 5x5 convolutions, two fully connected
# layers), its MNIST setting n = 16, B = 500, eta = 0.01, round trips
# 0.3 + 0.7 Exp(1); 28x28 synthetic images with MNIST-like sparsity.
C6 = DBWConfig(
    name="C6", model=CNN, n=16, B=500, d=784, C=10, H=500, S=60000, iters=20, eta=0.01,
    features="uniform", sparsity=0.8, seed=14696 + 6,
    times=TimeModel(kind="shifted_exp", shift=0.3, rate=1.0 / 0.7),
)

CONFIGS = {c.name: c for c in (C1, C2, C3, C4, C5, C6)}


def get(name: str) -> DBWConfig:
    return CONFIGS[name]


def describe(cfg: DBWConfig) -> str:
    tm = cfg.times
    return (f"{cfg.name}: {cfg.model} n={cfg.n} B={cfg.B} d={cfg.d} C={cfg.C}"
            + (f" H={cfg.H}" if cfg.model in (MLP, CNN) else "")
            + f" S={cfg.S} P={cfg.param_count} iters={cfg.iters} times={tm.kind}")
