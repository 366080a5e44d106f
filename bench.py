"""Benchmark of the DBW hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C5] [--no-cpu-baseline]

One step = one full DBW iteration (dbw_step): host time estimate, choice of
k, all n worker minibatch gradients, fastest-k aggregation, statistics, SGD
update and estimator bookkeeping.  Inputs are resident in HBM before the timed
region: the synthetic dataset, the per-iteration minibatch row indices and the
parameters; the per-iteration round-trip ticks are host arrays, as the
interface defines them.  Prints one JSON line.

Default workload: softmax regression with 256 workers x 512 rows, 3072
features (32x32x3-shaped) and 100 classes, the largest of the five workloads
(fp32 matrix-core bound).  The same line carries, under "hbm_roofline", the
bandwidth-bound workload (64 workers x 256 rows, 3072 features, 10 classes)
that the metric's %-of-peak-HBM figure refers to, and under "ps_kernels" the
aggregation and statistics calls at fixed k = n and ceil(n/2).

Order per workload: 0.1 s of untimed gradient launches (the GPU's clocks
settle only after some 40 ms of sustained load), the timed warm gradient
launches ("roofline"), the W untimed and K timed steps, a second pass of K
steps with per-launch events (the PS share), then the cold gradient launches
(each after a 1 GiB read that evicts the MALL).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "worker-gradient samples/sec per DBW iteration (1 MI355X); % peak HBM GB/s"
HBM_PEAK_GBS = 8000.0
MFMA_F32_PEAK_TFLOPS = 157.3   # dense fp32 matrix-core peak of the MI355X
FUSED_MAX_CLASSES = 16         # the single-pass softmax kernel covers C <= 16
FLUSH_BYTES = 1 << 30          # touched between launches for the cold figures (MALL is 256 MB)
SETTLE_S = 0.1                 # untimed gradient launches before the timed ones (clock settling)


TRAFFIC_FILE = {
    "C3": "profiles/traffic_worker_grads_softmax_n64_B256_d3072_C10.md",
    "C4": "profiles/traffic_worker_grads_mlp_n32_B64_784_512_10.md",
    "C5": "profiles/traffic_worker_grads_softmax_n256_B512_d3072_C100.md",
    "C6": "profiles/traffic_worker_grads_cnn_n16_B500_28x28_H500_C10.md",
}


def measured_traffic(cfg):
    """HBM bytes per gradient launch from the committed counter summary, or
    None when there is none for this workload or a kernel source it covers
    changed since it was taken."""
    import hashlib
    path = TRAFFIC_FILE.get(cfg.name)
    if not path or not os.path.exists(os.path.join(ROOT, path)):
        return None
    rec = None
    for line in open(os.path.join(ROOT, path)):
        if line.startswith("machine-readable:"):
            rec = json.loads(line.split(":", 1)[1])
    if rec is None:
        return None
    for src, digest in rec["kernel_sources_sha256"].items():
        with open(os.path.join(ROOT, src), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != digest:
                return None
    return rec["traffic_bytes_per_launch"]


def grads_bytes(cfg, P: int, gathered: bool) -> int:
    """Algorithmic bytes of one worker-gradient launch: every minibatch row
    and label read once, row indices, the parameters, and the n gradient rows
    and losses written."""
    rows = cfg.n * cfg.B
    return 4 * (rows * cfg.d + rows + (rows if gathered else 0) + P + cfg.n * P + cfg.n)


def grads_flops(cfg) -> float:
    """Useful fp32 flops of one worker-gradient launch (no padding): softmax
    logits X W and gradient X^T R; MLP hidden layer, head forward, head
    backward (dW2 and the hidden-unit residuals) and X^T dA.  CNN per image:
    both convolutions forward (24x24x20x25 and 8x8x50x500 products), the
    gradients of the conv2 filters and of its input and of the conv1 filters
    over the pooled-through positions only (one in four of each 2x2 window
    carries gradient), and the fully connected part forward and backward
    (3 x (800 H + H C) products)."""
    M = cfg.n * cfg.B
    if cfg.model == "softmax":
        return 4.0 * M * cfg.d * cfg.C
    if cfg.model == "cnn":
        c1 = 24 * 24 * 20 * 25
        c2 = 8 * 8 * 50 * 500
        macs = c1 + c2 + 2 * c2 / 4 + c1 / 4 + 3 * (800 * cfg.H + cfg.H * cfg.C)
        return 2.0 * M * macs
    return 4.0 * M * cfg.d * cfg.H + 6.0 * M * cfg.H * cfg.C


def roofline_bound(cfg) -> str:
    """The single-pass softmax kernel streams each row once and is bounded by
    HBM; the two-GEMM large-class path and the MLP are fp32 matrix-core work."""
    if cfg.model == "softmax" and cfg.C <= FUSED_MAX_CLASSES:
        return "hbm"
    return "mfma"


def grads_kernels(cfg) -> str:
    """The kernels one worker-gradient launch runs (names as in the traces)."""
    if cfg.model == "softmax":
        if cfg.C <= FUSED_MAX_CLASSES:
            return "k_softmax_mfma + k_slab_reduce_tiles"
        if cfg.C <= 112 and cfg.C % 4 == 0 and cfg.d % 4 == 0:
            return "k_logits_softmax_mfma + k_grads_mfma_n"
        return "k_logits_mfma + k_rows_softmax + k_grads_mfma"
    if cfg.model == "mlp":
        return "k_mlp_hidden_mfma + k_mlp_head + k_mlp_dw1_mfma (with the head's slab sums)"
    return "k_cnn_* + MLP kernels on the 800 features"


def step_bytes(cfg, P: int, k: int, gathered: bool) -> int:
    """Algorithmic bytes of one iteration: gradient launch, the k received
    gradient rows read once, parameters read and written, mean gradient
    written."""
    return grads_bytes(cfg, P, gathered) + 4 * (k * P + 3 * P)


def log(msg: str) -> None:
    """Progress on stderr (the JSON line is the only stdout output)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def workload_text(cfg) -> str:
    if cfg.model == "softmax":
        return (f"{cfg.name}: softmax regression, n={cfg.n} workers x B={cfg.B} rows, d={cfg.d}, C={cfg.C}, "
                f"minibatches gathered by index from a resident {cfg.S}x{cfg.d} dataset")
    if cfg.model == "mlp":
        return f"{cfg.name}: MLP {cfg.d}-{cfg.H}-{cfg.C}, n={cfg.n} workers x B={cfg.B} rows"
    return (f"{cfg.name}: CNN 28x28 conv5x5(20)-pool-conv5x5(50)-pool-FC{cfg.H}-FC{cfg.C}, "
            f"n={cfg.n} workers x B={cfg.B} images gathered from a resident {cfg.S}-image dataset")


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, timed on this host
def cpu_baseline(cfg, budget_s: float, budget_1core_s: float):
    """The float64 oracle on a bounded sample of the same workload: one
    untimed warm-up iteration (first touch of its buffers), then iterations
    until the budget is spent.  The time estimate (Eq. quadratic_opt) is
    solved outside the timed region and handed to the step, as the GPU
    figure excludes it too (the library solves it on a host thread that the
    device work hides).  BLAS threads are pinned to this process's cores;
    a second sample runs on one core."""
    from threadpoolctl import threadpool_info, threadpool_limits
    from dbw_inputs import gather, init_params
    from dbw_inputs import generate as gen
    from oracle import dbw as odbw

    cores = len(os.sched_getaffinity(0))
    X, y = gen.dataset(cfg)
    orc = odbw.DBWOracle(cfg, init_params(cfg))
    state = {"t": 0}

    def one(timed: bool) -> float:
        t = state["t"]
        idx = gen.batch_indices(cfg, t)
        Xt, yt = gather(X, y, idx)
        ticks = gen.round_trip_ticks(cfg, t)
        T_hat = orc.time_estimate()             # untimed, like the GPU figure
        t0 = time.perf_counter()
        orc.step(Xt, yt, ticks, T_hat=T_hat)
        state["t"] = t + 1
        return time.perf_counter() - t0

    def blas_threads():
        return max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])

    with threadpool_limits(limits=cores, user_api="blas"):
        used = blas_threads()
        one(False)                              # warm-up: first touch of the oracle's buffers
        first = state["t"]
        spent = 0.0
        while spent < budget_s or state["t"] == first:
            spent += one(True)
        done = state["t"] - first
    with threadpool_limits(limits=1, user_api="blas"):
        used1 = blas_threads()
        first1 = state["t"]
        spent1 = 0.0
        while spent1 < budget_1core_s or state["t"] == first1:
            spent1 += one(True)
        done1 = state["t"] - first1
    return {"value": cfg.n * cfg.B * done / spent, "unit": "samples/s", "cores": int(used),
            "kind": "oracle",
            "sample": f"iterations {first}..{first + done - 1} of {cfg.name} (iteration 0 untimed warm-up), "
                      f"float64 numpy oracle, time estimate solved outside the timed region, minibatch "
                      f"gather untimed, BLAS threads pinned to {used} with threadpoolctl, {spent:.1f} s",
            "value_1core": cfg.n * cfg.B * done1 / spent1,
            "sample_1core": f"the next iterations {first1}..{first1 + done1 - 1}, BLAS threads limited to "
                            f"{used1}, {spent1:.1f} s"}


# ---------------------------------------------------------------------------
# GPU measurements
class Workload:
    """Resident inputs and a context of one workload on the GPU."""

    def __init__(self, cfg, dev, n_iters: int):
        import torch
        import paper_2004_14696_amd as dbw
        from dbw_inputs import init_params
        from dbw_inputs import generate as gen
        self.cfg = cfg
        X, y = gen.dataset(cfg)
        self.Xd = torch.from_numpy(np.array(X)).to(dev)
        self.yd = torch.from_numpy(np.array(y)).to(dev)
        self.rows = [torch.from_numpy(gen.batch_indices(cfg, t)).to(dev) for t in range(n_iters)]
        self.ticks = [gen.round_trip_ticks(cfg, t) for t in range(n_iters)]
        self.w = torch.from_numpy(init_params(cfg)).to(dev)
        self.ctx = dbw.Context(dbw.config_from(cfg, S=cfg.S))
        self.P = self.ctx.P
        self.dev = dev

    def close(self):
        self.ctx.close()


def time_steps(wl, warmup: int, steps: int, timing_pass: bool):
    """Whole-job step timing (wall clock, host estimate included), then a
    pass with per-launch-group events for the PS share."""
    import torch
    import paper_2004_14696_amd as dbw
    ctx = wl.ctx
    for t in range(warmup):
        ctx.step(wl.w, wl.Xd, wl.yd, wl.ticks[t], rows=wl.rows[t], wait=False)
    ctx.sync()
    # timed region: host timers only (no device events in the launch stream)
    ctx.profile(2)
    ctx.profile_reset()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(ctx.stream)
    t1 = warmup + steps
    for t in range(warmup, t1):
        ctx.step(wl.w, wl.Xd, wl.yd, wl.ticks[t], rows=wl.rows[t], wait=False)
    ev1.record(ctx.stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ctx.sync()
    gpu_ms = ev0.elapsed_time(ev1)
    host = {g: ctx.kernel_time(getattr(dbw.binding, "DBW_KT_" + g))
            for g in ("HOST_ESTIMATE", "HOST_STEP", "HOST_WAIT", "HOST_QUEUE")}
    agg_ms = agg_n = choose_ms = choose_n = 0
    if timing_pass:
        ctx.profile(1)
        ctx.profile_reset()
        for t in range(t1, t1 + steps):
            ctx.step(wl.w, wl.Xd, wl.yd, wl.ticks[t], rows=wl.rows[t], wait=False)
        ctx.sync()
        agg_ms, agg_n = ctx.kernel_time(dbw.binding.DBW_KT_AGGREGATE)
        choose_ms, choose_n = ctx.kernel_time(dbw.binding.DBW_KT_CHOOSE)
    ctx.profile(False)
    st = ctx.export_state()
    return {"wall_ms": wall * 1e3 / steps, "gpu_ms": gpu_ms / steps,
            "agg_ms": agg_ms / steps if agg_n else None, "choose_ms": choose_ms / steps if choose_n else None,
            "host": {k: v[0] / max(v[1], 1) for k, v in host.items()}, "k_last": st["k_prev"]}


def time_grads_warm(wl, first: int, steps: int, settle_s: float = SETTLE_S):
    """The worker-gradient call (dbw_worker_grads) alone, warm: back to back
    between two events on the context stream, after untimed launches that
    keep the GPU busy for settle_s seconds (its clocks settle only after some
    40 ms of sustained load; from idle the first launches of the 256 x 512
    workload take 1.8 ms instead of 1.36).  Returns the mean launch time, the
    settling launches and their seconds, and the output buffers."""
    import torch
    ctx, cfg = wl.ctx, wl.cfg
    G = torch.empty((cfg.n, wl.P), dtype=torch.float32, device=wl.dev)
    Lb = torch.empty(cfg.n, dtype=torch.float32, device=wl.dev)
    settle = 0
    t0 = time.perf_counter()
    while True:
        for _ in range(4):
            ctx.worker_grads(wl.w, wl.Xd, wl.yd, rows=wl.rows[first + settle % steps], G=G, loss=Lb)
            settle += 1
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= settle_s:
            break
    settle_time = time.perf_counter() - t0
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g0.record(ctx.stream)
    for t in range(steps):
        ctx.worker_grads(wl.w, wl.Xd, wl.yd, rows=wl.rows[first + t], G=G, loss=Lb)
    g1.record(ctx.stream)
    torch.cuda.synchronize()
    return g0.elapsed_time(g1) / steps, settle, settle_time, G, Lb


def time_grads_cold(wl, first: int, steps: int, G, Lb):
    """The same call cold: each launch after a 1 GiB buffer was read
    (untimed), which evicts the 256 MB MALL and the L2s without leaving dirty
    lines behind, with events around the launch only."""
    import torch
    ctx = wl.ctx
    flush = torch.zeros(FLUSH_BYTES // 4, dtype=torch.float32, device=wl.dev)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for t in range(steps):
        flush.sum()                   # read-only: no dirty lines left to write back
        evs[t][0].record(ctx.stream)
        ctx.worker_grads(wl.w, wl.Xd, wl.yd, rows=wl.rows[first + t], G=G, loss=Lb)
        evs[t][1].record(ctx.stream)
    torch.cuda.synchronize()
    cold = sum(a.elapsed_time(b) for a, b in evs) / steps
    del flush
    ctx.sync()
    return cold


def roofline_block(cfg, P: int, warm_ms: float, cold_ms: float, launches: int) -> dict:
    gb = grads_bytes(cfg, P, True)
    bound = roofline_bound(cfg)
    if bound == "hbm":
        work, peak, unit = gb / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        work, peak, unit = grads_flops(cfg) / 1e12, MFMA_F32_PEAK_TFLOPS, "TFLOP/s"
    achieved = work / (warm_ms / 1e3)
    achieved_cold = work / (cold_ms / 1e3)
    return {
        "kernel": f"worker-gradient launch dbw_worker_grads ({grads_kernels(cfg)}); every G row written",
        "bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
        "traffic": measured_traffic(cfg), "bytes_per_launch": gb, "flops_per_launch": grads_flops(cfg),
        "avg_launch_ms": warm_ms, "launches": launches,
        "cold": {"avg_launch_ms": cold_ms, "achieved": achieved_cold, "frac": achieved_cold / peak,
                 "flush": "1 GiB device buffer read before each launch (untimed)"},
    }


def ps_fixed_k(wl, G, Lb, reps: int = 10):
    """The aggregation call (dbw_aggregate_fastest: rank selection, then the
    k rows streamed once into g) and the statistics call (dbw_grad_stats:
    the k rows listed from the mask and streamed against g, fixed-order
    finish) at
    fixed k = n and ceil(n/2) on the workload's gradient rows."""
    import torch
    ctx, cfg, P = wl.ctx, wl.cfg, wl.P
    n = cfg.n
    ticks = torch.from_numpy(np.ascontiguousarray(wl.ticks[0], dtype=np.int64)).to(wl.dev)
    g = torch.empty(P, dtype=torch.float32, device=wl.dev)
    mask = torch.empty(n, dtype=torch.uint8, device=wl.dev)
    sq = torch.empty(n, dtype=torch.float32, device=wl.dev)
    stats = torch.empty(4, dtype=torch.float64, device=wl.dev)
    out = []
    for k in (n, (n + 1) // 2):
        ctx.aggregate_fastest(G, ticks, k, g=g, mask=mask)
        ctx.grad_stats(G, mask, k, g, Lb, sqnorm=sq, stats=stats)
        ctx.sync()
        res = {"k": k}
        for name, fn, nbytes in (
                ("aggregate", lambda: ctx.aggregate_fastest(G, ticks, k, g=g, mask=mask),
                 4 * (k * P + P) + 9 * n),
                ("stats", lambda: ctx.grad_stats(G, mask, k, g, Lb, sqnorm=sq, stats=stats),
                 4 * (k * P + P) + 9 * n + 32)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(ctx.stream)
            for _ in range(reps):
                fn()
            e1.record(ctx.stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            gbs = nbytes / (ms / 1e3) / 1e9
            res[name] = {"ms": ms, "bytes": nbytes, "GB/s": gbs, "hbm_frac": gbs / HBM_PEAK_GBS}
        ctx.sync()
        out.append(res)
    return out


def measure(cfg, args, dev, with_ps: bool):
    total = args.warmup + 2 * args.steps + 1
    log(f"{cfg.name}: inputs")
    wl = Workload(cfg, dev, total)
    # the gradient launches first: their untimed settling launches bring the
    # GPU's clocks to their sustained level before the warm launches and the
    # steps are timed
    first = args.warmup + args.steps
    log(f"{cfg.name}: gradient launches, settling and warm")
    warm_ms, settle, settle_s, G, Lb = time_grads_warm(wl, first, args.steps)
    log(f"{cfg.name}: {args.warmup} + {args.steps} steps")
    st = time_steps(wl, args.warmup, args.steps, timing_pass=not args.no_kernel_timing)
    log(f"{cfg.name}: gradient launches, cold")
    cold_ms = time_grads_cold(wl, first, args.steps, G, Lb)
    res = {"step": st, "roofline": roofline_block(cfg, wl.P, warm_ms, cold_ms, args.steps), "P": wl.P}
    res["roofline"]["settle"] = {"launches": settle, "s": settle_s,
                                 "note": "untimed gradient launches before the warm launches and the steps"}
    if with_ps:
        log(f"{cfg.name}: aggregation and statistics at fixed k")
        res["ps_kernels"] = ps_fixed_k(wl, G, Lb)
    del G, Lb
    wl.close()
    return res


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="C5")
    ap.add_argument("--clock", choices=("fresh", "psw", "psi"), default="fresh",
                    help="virtual clock: every worker starts each iteration afresh, Push & Wait, "
                         "or Push & Interrupt")
    ap.add_argument("--policy", choices=("dbw", "static", "blind"), default="dbw",
                    help="choice of k: DBW, a static k (--k-static), or B-DBW (gain = k)")
    ap.add_argument("--k-static", type=int, default=0)
    ap.add_argument("--estimator", choices=("isotonic", "naive"), default="isotonic",
                    help="time estimate: constrained least squares, or the mean of cell (k,k)")
    ap.add_argument("--g-rows", choices=("all", "selected", "none"), default="none",
                    help="worker-gradient rows a step writes; with selected/none the selected "
                         "workers' slab partials are aggregated in one kernel where the softmax "
                         "kernel splits rows into slabs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--cpu-budget-1core", type=float, default=10.0)
    ap.add_argument("--no-extras", action="store_true",
                    help="only the named workload: no bandwidth-bound companion line, no fixed-k PS calls")
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="skip the per-launch-group event pass of the steps")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="for hardware-counter passes: three 256 MiB device copies (the calibration), "
                         "then five gradient launches of the workload; prints no bench line")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the DBW hot path here simulates all n workers on a single "
              f"MI355X; --gpus {args.gpus} is not supported.", file=sys.stderr)
        return 2

    import torch

    from dbw_inputs import get

    def configure(name):
        cfg = get(name)
        if args.clock != cfg.clock:
            cfg = cfg.replace(clock=args.clock)
        if args.policy == "static" and not 1 <= args.k_static <= cfg.n:
            sys.exit(f"--policy static needs --k-static in [1, {cfg.n}]")
        return cfg.replace(policy=args.policy, k_static=args.k_static if args.policy == "static" else 0,
                           estimator=args.estimator, g_rows=args.g_rows)

    cfg = configure(args.workload)
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    if args.traffic_probe:
        src = torch.full((64 * 1024 * 1024,), 1.0, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        wl = Workload(cfg, dev, 5)
        G = torch.empty((cfg.n, wl.P), dtype=torch.float32, device=dev)
        Lb = torch.empty(cfg.n, dtype=torch.float32, device=dev)
        for t in range(5):
            wl.ctx.worker_grads(wl.w, wl.Xd, wl.yd, rows=wl.rows[t], G=G, loss=Lb)
        wl.ctx.sync()
        print(f"traffic probe: 3 copies of 256 MiB, 5 gradient launches of {cfg.name}", flush=True)
        return 0

    extras = not args.no_extras and args.workload == "C5"
    main_res = measure(cfg, args, dev, with_ps=extras)
    st = main_res["step"]
    P = main_res["P"]
    ms_per_step = st["wall_ms"]     # whole job: host estimate, launches, device work
    value = cfg.n * cfg.B / (ms_per_step / 1e3)
    sb = step_bytes(cfg, P, st["k_last"], True)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": workload_text(cfg),
            "n": cfg.n, "B": cfg.B, "d": cfg.d, "C": cfg.C, "H": cfg.H, "P": P, "clock": cfg.clock,
            "policy": cfg.policy, "k_static": cfg.k_static, "estimator": cfg.estimator, "g_rows": cfg.g_rows,
        },
        "roofline": main_res["roofline"],
        "step": {
            "gpu_ms_per_step": st["gpu_ms"],
            "wall_ms_per_step": st["wall_ms"],
            "bytes_per_step": sb,
            "hbm_frac": sb / (ms_per_step / 1e3) / 1e9 / HBM_PEAK_GBS,
            "aggregate_and_stats_ms_per_step": st["agg_ms"],
            "choose_ms_per_step": st["choose_ms"],
            "host_estimate_ms_per_step": st["host"]["HOST_ESTIMATE"],
            "host_step_call_ms": st["host"]["HOST_STEP"],
            "host_wait_for_estimate_ms": st["host"]["HOST_WAIT"],
            "host_queue_ms": st["host"]["HOST_QUEUE"],
            "k_last": st["k_last"],
        },
    }
    if extras:
        out["ps_kernels"] = {
            "workload": cfg.name,
            "calls": main_res["ps_kernels"],
            "note": "whole calls by HIP events (rank selection or mask-to-list, the streaming kernel, "
                    "and for the statistics the fixed-order finish); bytes = the k rows read once, g "
                    "written or read, ticks/mask/loss/sqnorm",
        }
        c3 = configure("C3")
        r3 = measure(c3, args, dev, with_ps=False)
        s3 = r3["step"]
        out["hbm_roofline"] = {
            "workload": workload_text(c3),
            **r3["roofline"],
            "step_ms": s3["wall_ms"],
            "step_samples_per_s": c3.n * c3.B / (s3["wall_ms"] / 1e3),
            "g_rows": c3.g_rows,
            "k_last": s3["k_last"],
        }
    if not args.no_cpu_baseline:
        log(f"{cfg.name}: CPU baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_budget, args.cpu_budget_1core)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
