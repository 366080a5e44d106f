"""CPU oracle of the Dynamic Backup Workers (DBW) iteration -- TEST INFRASTRUCTURE.

A plain, slow, float64 implementation of what one DBW parameter-server
iteration computes, written from the paper's definitions (Xu, Neglia,
Sebastianelli, "Dynamic Backup Workers for Parallel Machine Learning"):

* ``model``          -- worker minibatch gradients and losses (Sect. 2, Eq. gradient)
* ``ps``             -- fastest-k selection, averaging (Eq. grad_bw), the
                        end-of-iteration estimators (Eqs. sumvariancekt,
                        normsquarekt, estimateL) and the SGD update (Eq. update)
* ``time_estimator`` -- the constrained least-squares estimate of the
                        order-statistic times (Sect. 3.2, Eq. quadratic_opt)
* ``dbw``            -- the D-window averages (Eqs. varianceoverD,
                        normsquareoverD, LoverD), the gain (Eq. gain), the
                        choice of k (Eqs. greedy, greedy2) and the full
                        iteration with its bookkeeping.

This package is the reference the GPU library is checked against.  Only the
test-suite, the smoke check and the benchmark's CPU-baseline leg may import
it; the product path never does.  It shares no code with the HIP library and
imports nothing from it.
"""
from . import dbw, model, ps, time_estimator  # noqa: F401
from .dbw import DBWOracle, choose_k, window_mean  # noqa: F401
from .model import mlp_worker_grads, softmax_worker_grads  # noqa: F401
from .ps import aggregate, grad_stats, select_fastest, sgd_update  # noqa: F401
from .time_estimator import fit_observed, time_estimate  # noqa: F401
