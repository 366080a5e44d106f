"""ctypes binding of libdbw.so (the C ABI declared in include/dbw.h).

Argument marshalling only: every step of the DBW iteration runs in the HIP
library.  PyTorch supplies device memory and the stream; tensors are checked
for dtype, device, contiguity and shape before their pointers are passed.
The binding fails loudly when the library is not built -- there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_int32, c_int64, c_size_t, c_uint8, c_void_p

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdbw.so")

DBW_OK, DBW_EINVAL, DBW_ERANGE, DBW_EHIP, DBW_ESTATE, DBW_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
DBW_SOFTMAX, DBW_MLP, DBW_CNN = 0, 1, 2
DBW_CLOCK_FRESH, DBW_CLOCK_PSW, DBW_CLOCK_PSI = 0, 1, 2
DBW_POLICY_DBW, DBW_POLICY_STATIC, DBW_POLICY_BLIND = 0, 1, 2
DBW_ESTIMATOR_ISOTONIC, DBW_ESTIMATOR_NAIVE = 0, 1
DBW_G_ROWS_ALL, DBW_G_ROWS_SELECTED, DBW_G_ROWS_NONE = 0, 1, 2
DBW_MAX_N, DBW_MAX_D = 1024, 64
DBW_KT_GRADS, DBW_KT_AGGREGATE, DBW_KT_CHOOSE, DBW_KT_HOST_ESTIMATE, DBW_KT_HOST_STEP = 0, 1, 2, 3, 4
DBW_KT_HOST_WAIT, DBW_KT_HOST_QUEUE = 5, 6

STATUS_NAMES = {0: "DBW_OK", -1: "DBW_EINVAL", -2: "DBW_ERANGE", -3: "DBW_EHIP",
                -4: "DBW_ESTATE", -5: "DBW_EUNSUPPORTED"}

EXPORTED = (
    "dbw_param_count", "dbw_create", "dbw_destroy", "dbw_last_error", "dbw_sync",
    "dbw_worker_grads", "dbw_aggregate_fastest", "dbw_grad_stats", "dbw_choose_b", "dbw_step",
    "dbw_step_outputs", "dbw_time_estimate", "dbw_state_export", "dbw_state_import",
    "dbw_samples_export", "dbw_samples_import", "dbw_profile_enable", "dbw_kernel_time",
    "dbw_profile_reset", "dbw_time_estimator_create", "dbw_time_estimator_destroy",
    "dbw_time_estimator_solve", "dbw_time_estimator_stats", "dbw_busy_export", "dbw_busy_import",
    "dbw_grad_stats_static",
)
DBW_STATIC_SCRATCH_BYTES = 8 * 1024 * 1024


class DBWError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [("model", c_int32), ("n", c_int32), ("B", c_int32), ("d", c_int32),
                ("C", c_int32), ("H", c_int32), ("D", c_int32), ("clock", c_int32),
                ("policy", c_int32), ("k_static", c_int32), ("estimator", c_int32),
                ("g_rows", c_int32), ("eta", c_double), ("beta", c_double), ("S", c_int64)]


class IterStats(ctypes.Structure):
    _fields_ = [("gnorm2", c_double), ("V_plus", c_double), ("N_plus", c_double), ("F_hat", c_double)]


class EstimatorState(ctypes.Structure):
    _fields_ = [("t", c_int64), ("k_prev", c_int32), ("nV", c_int32), ("nL", c_int32),
                ("nF", c_int32), ("F_prev", c_double), ("F_prev2", c_double),
                ("hV", c_double * DBW_MAX_D), ("hN", c_double * DBW_MAX_D),
                ("hL", c_double * DBW_MAX_D)]


class StepBuffers(ctypes.Structure):
    _fields_ = [(name, c_void_p) for name in
                ("G", "loss", "g", "mask", "sqnorm", "stats", "T_hat", "objective", "k", "b")]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libdbw.so and declare its prototypes (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2004_14696_amd.build`")
    # torch carries its own HIP runtime; loaded first, it is the one the
    # library binds to (loaded after the library, it would be a second
    # runtime in the process, and device memory and streams would not be
    # shared between the two)
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    st = c_int32
    P = c_void_p
    lib.dbw_param_count.argtypes = [POINTER(Config)]
    lib.dbw_param_count.restype = c_int64
    lib.dbw_create.argtypes = [POINTER(Config), P, POINTER(P)]
    lib.dbw_create.restype = st
    lib.dbw_destroy.argtypes = [P]
    lib.dbw_destroy.restype = None
    lib.dbw_last_error.argtypes = [P]
    lib.dbw_last_error.restype = ctypes.c_char_p
    lib.dbw_sync.argtypes = [P]
    lib.dbw_sync.restype = st
    lib.dbw_worker_grads.argtypes = [P, P, P, P, P, P, P]
    lib.dbw_worker_grads.restype = st
    lib.dbw_aggregate_fastest.argtypes = [P, P, P, c_int32, P, P]
    lib.dbw_aggregate_fastest.restype = st
    lib.dbw_grad_stats.argtypes = [P, P, P, c_int32, P, P, P, P]
    lib.dbw_grad_stats.restype = st
    lib.dbw_choose_b.argtypes = [P, P, P, P, P]
    lib.dbw_choose_b.restype = st
    lib.dbw_step.argtypes = [P, P, P, P, P, POINTER(c_int64), POINTER(c_int32)]
    lib.dbw_step.restype = st
    lib.dbw_step_outputs.argtypes = [P, POINTER(StepBuffers)]
    lib.dbw_step_outputs.restype = st
    lib.dbw_time_estimate.argtypes = [c_int32, POINTER(c_int64), POINTER(c_int64), POINTER(c_double)]
    lib.dbw_time_estimate.restype = st
    lib.dbw_time_estimator_create.argtypes = [POINTER(P)]
    lib.dbw_time_estimator_create.restype = st
    lib.dbw_time_estimator_destroy.argtypes = [P]
    lib.dbw_time_estimator_destroy.restype = None
    lib.dbw_time_estimator_solve.argtypes = [P, c_int32, POINTER(c_int64), POINTER(c_int64), POINTER(c_double)]
    lib.dbw_time_estimator_solve.restype = st
    lib.dbw_time_estimator_stats.argtypes = [P, POINTER(c_int64), POINTER(c_int64), POINTER(c_int64)]
    lib.dbw_time_estimator_stats.restype = st
    lib.dbw_busy_export.argtypes = [P, POINTER(c_int64)]
    lib.dbw_busy_export.restype = st
    lib.dbw_busy_import.argtypes = [P, POINTER(c_int64)]
    lib.dbw_busy_import.restype = st
    lib.dbw_state_export.argtypes = [P, POINTER(EstimatorState)]
    lib.dbw_state_export.restype = st
    lib.dbw_state_import.argtypes = [P, POINTER(EstimatorState)]
    lib.dbw_state_import.restype = st
    lib.dbw_samples_export.argtypes = [P, POINTER(c_int64), POINTER(c_int64), POINTER(c_int64)]
    lib.dbw_samples_export.restype = st
    lib.dbw_samples_import.argtypes = [P, POINTER(c_int64), POINTER(c_int64), c_int64]
    lib.dbw_samples_import.restype = st
    lib.dbw_profile_enable.argtypes = [P, c_int32]
    lib.dbw_profile_enable.restype = st
    lib.dbw_kernel_time.argtypes = [P, c_int32, POINTER(c_double), POINTER(c_int64)]
    lib.dbw_kernel_time.restype = st
    lib.dbw_profile_reset.argtypes = [P]
    lib.dbw_profile_reset.restype = st
    lib.dbw_grad_stats_static.argtypes = [c_int32, c_int64, P, P, c_int32, P, P, c_double, P, P, P]
    lib.dbw_grad_stats_static.restype = st
    _lib = lib
    return lib


CLOCKS = {"fresh": DBW_CLOCK_FRESH, "psw": DBW_CLOCK_PSW, "psi": DBW_CLOCK_PSI}
POLICIES = {"dbw": DBW_POLICY_DBW, "static": DBW_POLICY_STATIC, "blind": DBW_POLICY_BLIND}
ESTIMATORS = {"isotonic": DBW_ESTIMATOR_ISOTONIC, "naive": DBW_ESTIMATOR_NAIVE}
G_ROWS = {"all": DBW_G_ROWS_ALL, "selected": DBW_G_ROWS_SELECTED, "none": DBW_G_ROWS_NONE}


def make_config(model: str | int, n: int, B: int, d: int, C: int, H: int = 0, eta: float = 0.1,
                beta: float = 1.01, D: int = 5, S: int = 0, clock: str | int = DBW_CLOCK_FRESH,
                policy: str | int = DBW_POLICY_DBW, k_static: int = 0,
                estimator: str | int = DBW_ESTIMATOR_ISOTONIC, g_rows: str | int = DBW_G_ROWS_ALL) -> Config:
    if isinstance(model, str):
        model = {"softmax": DBW_SOFTMAX, "mlp": DBW_MLP, "cnn": DBW_CNN}[model]
    if isinstance(clock, str):
        clock = CLOCKS[clock]
    if isinstance(policy, str):
        policy = POLICIES[policy]
    if isinstance(estimator, str):
        estimator = ESTIMATORS[estimator]
    if isinstance(g_rows, str):
        g_rows = G_ROWS[g_rows]
    return Config(model=model, n=n, B=B, d=d, C=C, H=H, D=D, clock=clock, policy=policy,
                  k_static=k_static, estimator=estimator, g_rows=g_rows, eta=eta, beta=beta, S=S)


def param_count(cfg: Config) -> int:
    return int(load_library().dbw_param_count(ctypes.byref(cfg)))


def time_estimate(cnt, tsum) -> np.ndarray:
    """Host time estimate (dbw_time_estimate): T_hat[k-1] for k = 1..n (NaN
    where no estimate exists)."""
    lib = load_library()
    cnt = np.ascontiguousarray(cnt, dtype=np.int64)
    tsum = np.ascontiguousarray(tsum, dtype=np.int64)
    n = cnt.shape[0]
    if cnt.shape != (n, n) or tsum.shape != (n, n):
        raise ValueError("cnt and tsum must be n x n")
    out = np.empty(n, dtype=np.float64)
    s = lib.dbw_time_estimate(n, cnt.ctypes.data_as(POINTER(c_int64)),
                              tsum.ctypes.data_as(POINTER(c_int64)),
                              out.ctypes.data_as(POINTER(c_double)))
    if s != DBW_OK:
        raise DBWError(s, "dbw_time_estimate rejected its input")
    return out


class TimeEstimator:
    """Incremental exact time estimate (dbw_time_estimator_*)."""

    def __init__(self):
        self.lib = load_library()
        h = c_void_p()
        s = self.lib.dbw_time_estimator_create(ctypes.byref(h))
        if s != DBW_OK:
            raise DBWError(s, "dbw_time_estimator_create failed")
        self.h = h

    def solve(self, cnt, tsum) -> np.ndarray:
        cnt = np.ascontiguousarray(cnt, dtype=np.int64)
        tsum = np.ascontiguousarray(tsum, dtype=np.int64)
        n = cnt.shape[0]
        if cnt.shape != (n, n) or tsum.shape != (n, n):
            raise ValueError("cnt and tsum must be n x n")
        out = np.empty(n, dtype=np.float64)
        s = self.lib.dbw_time_estimator_solve(self.h, n, cnt.ctypes.data_as(POINTER(c_int64)),
                                              tsum.ctypes.data_as(POINTER(c_int64)),
                                              out.ctypes.data_as(POINTER(c_double)))
        if s != DBW_OK:
            raise DBWError(s, "dbw_time_estimator_solve rejected its input")
        return out

    def stats(self) -> dict:
        """Solves so far by path: fast (per-column fit feasible), warm, full."""
        f, w, u = c_int64(), c_int64(), c_int64()
        s = self.lib.dbw_time_estimator_stats(self.h, ctypes.byref(f), ctypes.byref(w), ctypes.byref(u))
        if s != DBW_OK:
            raise DBWError(s, "dbw_time_estimator_stats failed")
        return {"fast": f.value, "warm": w.value, "full": u.value}

    def __del__(self):
        if getattr(self, "h", None):
            self.lib.dbw_time_estimator_destroy(self.h)
            self.h = None


def grad_stats_static(G, mask, k, g, loss, V_window=0.0, sqnorm=None, stats=None, stream=None):
    """dbw_grad_stats_static: the statistics of dbw_grad_stats with no context
    and no allocation inside the call (scratch in the library's static device
    array).  G [n][P] float32, mask [n] uint8, g [P] float32, loss [n]
    float32, all on the current device; V_window is V_plus for k = 1.
    Returns (sqnorm [n] float32, stats float64 [4] = gnorm2, V_plus, N_plus,
    F_hat); pass sqnorm and stats to write into existing tensors."""
    torch = _torch()
    lib = load_library()
    if G.dim() != 2:
        raise ValueError("G must be [n][P]")
    n, P = G.shape
    dev = G.device
    for name, t, dtype, shape in (("G", G, torch.float32, (n, P)), ("mask", mask, torch.uint8, (n,)),
                                  ("g", g, torch.float32, (P,)), ("loss", loss, torch.float32, (n,))):
        if t.device != dev or t.dtype != dtype or not t.is_contiguous() or tuple(t.shape) != shape:
            raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {shape} on {dev}")
    sqnorm = torch.empty(n, dtype=torch.float32, device=dev) if sqnorm is None else sqnorm
    stats = torch.empty(4, dtype=torch.float64, device=dev) if stats is None else stats
    if tuple(sqnorm.shape) != (n,) or sqnorm.dtype != torch.float32 or sqnorm.device != dev:
        raise ValueError("sqnorm must be float32 [n] on the device of G")
    if tuple(stats.shape) != (4,) or stats.dtype != torch.float64 or stats.device != dev:
        raise ValueError("stats must be float64 [4] on the device of G")
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    s = lib.dbw_grad_stats_static(int(n), int(P), c_void_p(G.data_ptr()), c_void_p(mask.data_ptr()), int(k),
                                  c_void_p(g.data_ptr()), c_void_p(loss.data_ptr()), float(V_window),
                                  c_void_p(sqnorm.data_ptr()), c_void_p(stats.data_ptr()),
                                  c_void_p(stream.cuda_stream))
    if s != DBW_OK:
        raise DBWError(s, lib.dbw_last_error(None).decode())
    return sqnorm, stats


# ---------------------------------------------------------------------------
_hip = None


def _hip_runtime():
    """libamdhip64 for device-to-device copies out of the library's buffers."""
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpyAsync.argtypes = [c_void_p, c_void_p, c_size_t, c_int32, c_void_p]
        _hip.hipMemcpyAsync.restype = c_int32
    return _hip


HIP_MEMCPY_D2D = 3


def _torch():
    import torch
    return torch


class Context:
    """One DBW parameter-server simulation bound to a torch CUDA (HIP) stream."""

    def __init__(self, cfg: Config, stream=None, device=None):
        torch = _torch()
        self.lib = load_library()
        self.cfg = cfg
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None else device)
        with torch.cuda.device(self.device):
            self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
            handle = c_void_p()
            s = self.lib.dbw_create(ctypes.byref(cfg), c_void_p(self.stream.cuda_stream), ctypes.byref(handle))
        if s != DBW_OK:
            raise DBWError(s, "dbw_create failed (invalid configuration or HIP error)")
        self.h = handle
        self.P = param_count(cfg)

    def close(self):
        if getattr(self, "h", None):
            self.lib.dbw_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- helpers -------------------------------------------------------------
    def _check(self, s: int, what: str):
        if s != DBW_OK:
            raise DBWError(s, f"{what}: {self.lib.dbw_last_error(self.h).decode()}")

    def _dev(self, t, dtype, shape, name):
        torch = _torch()
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch tensor")
        if t.device != self.device:
            raise ValueError(f"{name} must live on {self.device}, not {t.device}")
        if t.dtype != dtype:
            raise ValueError(f"{name} must be {dtype}, not {t.dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if shape is not None and tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, not {tuple(t.shape)}")
        return c_void_p(t.data_ptr())

    def _empty(self, shape, dtype):
        return _torch().empty(shape, dtype=dtype, device=self.device)

    def _batch(self, X, y, rows):
        torch = _torch()
        c = self.cfg
        if rows is None:
            return (self._dev(X, torch.float32, (c.n, c.B, c.d), "X"),
                    self._dev(y, torch.int32, (c.n, c.B), "y"), None)
        return (self._dev(X, torch.float32, (c.S, c.d), "X (dataset)"),
                self._dev(y, torch.int32, (c.S,), "y (labels)"),
                self._dev(rows, torch.int32, (c.n, c.B), "rows"))

    # -- the five calls --------------------------------------------------------
    def worker_grads(self, w, X, y, rows=None, G=None, loss=None):
        torch = _torch()
        c = self.cfg
        G = self._empty((c.n, self.P), torch.float32) if G is None else G
        loss = self._empty((c.n,), torch.float32) if loss is None else loss
        px, py, pr = self._batch(X, y, rows)
        self._check(self.lib.dbw_worker_grads(self.h, self._dev(w, torch.float32, (self.P,), "w"), px, py, pr,
                                              self._dev(G, torch.float32, (c.n, self.P), "G"),
                                              self._dev(loss, torch.float32, (c.n,), "loss")),
                    "dbw_worker_grads")
        return G, loss

    def aggregate_fastest(self, G, ticks, k, g=None, mask=None):
        torch = _torch()
        c = self.cfg
        g = self._empty((self.P,), torch.float32) if g is None else g
        mask = self._empty((c.n,), torch.uint8) if mask is None else mask
        self._check(self.lib.dbw_aggregate_fastest(
            self.h, self._dev(G, torch.float32, (c.n, self.P), "G"),
            self._dev(ticks, torch.int64, (c.n,), "ticks"), int(k),
            self._dev(g, torch.float32, (self.P,), "g"), self._dev(mask, torch.uint8, (c.n,), "mask")),
            "dbw_aggregate_fastest")
        return g, mask

    def grad_stats(self, G, mask, k, g, loss, sqnorm=None, stats=None):
        """Returns (sqnorm [n] float32, stats float64 [4] = gnorm2, V_plus, N_plus, F_hat)."""
        torch = _torch()
        c = self.cfg
        sqnorm = self._empty((c.n,), torch.float32) if sqnorm is None else sqnorm
        stats = self._empty((4,), torch.float64) if stats is None else stats
        self._check(self.lib.dbw_grad_stats(
            self.h, self._dev(G, torch.float32, (c.n, self.P), "G"),
            self._dev(mask, torch.uint8, (c.n,), "mask"), int(k),
            self._dev(g, torch.float32, (self.P,), "g"), self._dev(loss, torch.float32, (c.n,), "loss"),
            self._dev(sqnorm, torch.float32, (c.n,), "sqnorm"), self._dev(stats, torch.float64, (4,), "stats")),
            "dbw_grad_stats")
        return sqnorm, stats

    def choose_b(self, T_hat, k=None, b=None, objective=None):
        torch = _torch()
        c = self.cfg
        k = self._empty((1,), torch.int32) if k is None else k
        b = self._empty((1,), torch.int32) if b is None else b
        objective = self._empty((c.n,), torch.float64) if objective is None else objective
        self._check(self.lib.dbw_choose_b(self.h, self._dev(T_hat, torch.float64, (c.n,), "T_hat"),
                                          self._dev(k, torch.int32, (1,), "k"),
                                          self._dev(b, torch.int32, (1,), "b"),
                                          self._dev(objective, torch.float64, (c.n,), "objective")),
                    "dbw_choose_b")
        return k, b, objective

    def step(self, w, X, y, ticks, rows=None, wait: bool = False):
        """One DBW iteration; updates w in place.  Returns k_t if ``wait``."""
        torch = _torch()
        c = self.cfg
        ticks = np.ascontiguousarray(ticks, dtype=np.int64)
        if ticks.shape != (c.n,):
            raise ValueError(f"ticks must have shape ({c.n},)")
        px, py, pr = self._batch(X, y, rows)
        kout = c_int32(0)
        self._check(self.lib.dbw_step(self.h, self._dev(w, torch.float32, (self.P,), "w"), px, py, pr,
                                      ticks.ctypes.data_as(POINTER(c_int64)),
                                      ctypes.byref(kout) if wait else None), "dbw_step")
        return int(kout.value) if wait else None

    def step_outputs(self):
        """Copies of the buffers the last step wrote (torch tensors)."""
        torch = _torch()
        c = self.cfg
        bufs = StepBuffers()
        self._check(self.lib.dbw_step_outputs(self.h, ctypes.byref(bufs)), "dbw_step_outputs")
        spec = {"G": ((c.n, self.P), torch.float32), "loss": ((c.n,), torch.float32),
                "g": ((self.P,), torch.float32), "mask": ((c.n,), torch.uint8),
                "sqnorm": ((c.n,), torch.float32), "stats": ((4,), torch.float64),
                "T_hat": ((c.n,), torch.float64), "objective": ((c.n,), torch.float64),
                "k": ((1,), torch.int32), "b": ((1,), torch.int32)}
        hip = _hip_runtime()
        out = {}
        for name, (shape, dtype) in spec.items():
            t = self._empty(shape, dtype)
            nbytes = t.numel() * t.element_size()
            e = hip.hipMemcpyAsync(c_void_p(t.data_ptr()), c_void_p(getattr(bufs, name)), nbytes,
                                   HIP_MEMCPY_D2D, c_void_p(self.stream.cuda_stream))
            if e != 0:
                raise DBWError(DBW_EHIP, f"hipMemcpyAsync of {name} failed ({e})")
            out[name] = t
        return out

    def sync(self):
        self._check(self.lib.dbw_sync(self.h), "dbw_sync")

    # -- state -------------------------------------------------------------------
    def export_state(self) -> dict:
        s = EstimatorState()
        self._check(self.lib.dbw_state_export(self.h, ctypes.byref(s)), "dbw_state_export")
        return {"t": s.t, "k_prev": s.k_prev, "hV": list(s.hV[:s.nV]), "hN": list(s.hN[:s.nV]),
                "hL": list(s.hL[:s.nL]), "nF": s.nF, "F_prev": s.F_prev, "F_prev2": s.F_prev2}

    def import_state(self, st: dict):
        s = EstimatorState()
        s.t = int(st["t"])
        s.k_prev = int(st["k_prev"])
        hV, hN, hL = list(st["hV"]), list(st["hN"]), list(st["hL"])
        if len(hV) != len(hN):
            raise ValueError("hV and hN must have the same length")
        s.nV, s.nL, s.nF = len(hV), len(hL), int(st["nF"])
        for i, v in enumerate(hV):
            s.hV[i] = v
        for i, v in enumerate(hN):
            s.hN[i] = v
        for i, v in enumerate(hL):
            s.hL[i] = v
        s.F_prev = float(st.get("F_prev", 0.0))
        s.F_prev2 = float(st.get("F_prev2", 0.0))
        self._check(self.lib.dbw_state_import(self.h, ctypes.byref(s)), "dbw_state_import")

    def export_samples(self):
        n = self.cfg.n
        cnt = np.zeros((n, n), np.int64)
        tsum = np.zeros((n, n), np.int64)
        clock = c_int64(0)
        self._check(self.lib.dbw_samples_export(self.h, cnt.ctypes.data_as(POINTER(c_int64)),
                                                tsum.ctypes.data_as(POINTER(c_int64)), ctypes.byref(clock)),
                    "dbw_samples_export")
        return cnt, tsum, int(clock.value)

    def export_busy(self) -> np.ndarray:
        """Push & Wait: the time each worker becomes free (ticks)."""
        out = np.empty(self.cfg.n, dtype=np.int64)
        self._check(self.lib.dbw_busy_export(self.h, out.ctypes.data_as(POINTER(c_int64))), "dbw_busy_export")
        return out

    def import_busy(self, busy):
        b = np.ascontiguousarray(busy, dtype=np.int64)
        if b.shape != (self.cfg.n,):
            raise ValueError(f"busy must have shape ({self.cfg.n},)")
        self._check(self.lib.dbw_busy_import(self.h, b.ctypes.data_as(POINTER(c_int64))), "dbw_busy_import")

    def import_samples(self, cnt, tsum, clock: int = 0):
        cnt = np.ascontiguousarray(cnt, dtype=np.int64)
        tsum = np.ascontiguousarray(tsum, dtype=np.int64)
        self._check(self.lib.dbw_samples_import(self.h, cnt.ctypes.data_as(POINTER(c_int64)),
                                                tsum.ctypes.data_as(POINTER(c_int64)), int(clock)),
                    "dbw_samples_import")

    # -- timing --------------------------------------------------------------------
    def profile(self, on=True):
        """True/1: device events and host timers; 2: host timers only; False/0: off."""
        mode = 1 if on is True else (0 if on is False else int(on))
        self._check(self.lib.dbw_profile_enable(self.h, mode), "dbw_profile_enable")

    def profile_reset(self):
        self._check(self.lib.dbw_profile_reset(self.h), "dbw_profile_reset")

    def kernel_time(self, group: int):
        ms, n = c_double(0.0), c_int64(0)
        self._check(self.lib.dbw_kernel_time(self.h, int(group), ctypes.byref(ms), ctypes.byref(n)),
                    "dbw_kernel_time")
        return float(ms.value), int(n.value)
