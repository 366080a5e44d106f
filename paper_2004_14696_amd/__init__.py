"""MI355X-native hot path of Dynamic Backup Workers (DBW).

A synchronous parameter server with n logical workers simulated on one GPU:
worker minibatch gradients, aggregation of the fastest k, gradient
statistics, the DBW choice of k and the SGD update, all in hand-written HIP
kernels for gfx950 behind the C ABI of ``include/dbw.h``.  This package is
the Python binding of that library.
"""
from .binding import (DBW_MLP, DBW_SOFTMAX, Config, Context, DBWError, load_library,  # noqa: F401
                      make_config, param_count, time_estimate)

__all__ = ["Config", "Context", "DBWError", "load_library", "make_config", "param_count",
           "time_estimate", "DBW_SOFTMAX", "DBW_MLP", "config_from"]


def config_from(wl, S: int = 0) -> Config:
    """C-ABI configuration for a workload description (dbw_inputs.DBWConfig)."""
    return make_config(wl.model, wl.n, wl.B, wl.d, wl.C, wl.H, eta=wl.eta, beta=wl.beta, D=wl.D, S=S,
                       clock=getattr(wl, "clock", "fresh"), policy=getattr(wl, "policy", "dbw"),
                       k_static=getattr(wl, "k_static", 0), estimator=getattr(wl, "estimator", "isotonic"),
                       g_rows=getattr(wl, "g_rows", "all"))
