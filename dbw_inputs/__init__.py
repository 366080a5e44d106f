"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

Holds workload descriptions and random draws only; none of the DBW method's
arithmetic lives here.
"""
from .configs import (C1, C2, C3, C4, C5, C6, CNN, CONFIGS, MLP, SOFTMAX, TICKS_PER_UNIT,
                      DBWConfig, TimeModel, describe, get)
from .generate import (batch_indices, dataset, gather, init_params, iteration_inputs,
                       round_trip_ticks, round_trip_times)

__all__ = [
    "C1", "C2", "C3", "C4", "C5", "C6", "CNN", "CONFIGS", "MLP", "SOFTMAX", "TICKS_PER_UNIT",
    "DBWConfig", "TimeModel", "describe", "get", "batch_indices", "dataset",
    "gather", "init_params", "iteration_inputs", "round_trip_ticks", "round_trip_times",
]
