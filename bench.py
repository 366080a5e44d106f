"""Benchmark of the DBW hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C3] [--no-cpu-baseline]

One step = one full DBW iteration (dbw_step): host time estimate, choice of
k, all n worker minibatch gradients, fastest-k aggregation, statistics, SGD
update and estimator bookkeeping.  Inputs are resident in HBM before the timed
region: the synthetic dataset, the per-iteration minibatch row indices and the
parameters; the per-iteration round-trip ticks are host arrays, as the
interface defines them.  Prints one JSON line.

Default workload: softmax regression with 64 workers x 256 rows, 3072
features (32x32x3-shaped) and 10 classes -- the bandwidth-bound workload the
metric's %-of-peak-HBM figure refers to.
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
    import os
    path = TRAFFIC_FILE.get(cfg.name)
    root = os.path.dirname(os.path.abspath(__file__))
    if not path or not os.path.exists(os.path.join(root, path)):
        return None
    rec = None
    for line in open(os.path.join(root, path)):
        if line.startswith("machine-readable:"):
            rec = json.loads(line.split(":", 1)[1])
    if rec is None:
        return None
    for src, digest in rec["kernel_sources_sha256"].items():
        with open(os.path.join(root, src), "rb") as f:
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


def step_bytes(cfg, P: int, k: int, gathered: bool) -> int:
    """Algorithmic bytes of one iteration: gradient launch, the k received
    gradient rows read once, parameters read and written, mean gradient
    written."""
    return grads_bytes(cfg, P, gathered) + 4 * (k * P + 3 * P)


def cpu_baseline(cfg, iters_cap: int, budget_s: float):
    """The oracle timed on this host on the first iterations of the same
    workload (bounded sample)."""
    from dbw_inputs import gather, init_params
    from dbw_inputs import generate as gen
    from oracle import dbw as odbw
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    X, y = gen.dataset(cfg)
    orc = odbw.DBWOracle(cfg, init_params(cfg))
    done, spent = 0, 0.0
    while done < iters_cap and spent < budget_s:
        idx = gen.batch_indices(cfg, done)
        Xt, yt = gather(X, y, idx)
        ticks = gen.round_trip_ticks(cfg, done)
        t0 = time.perf_counter()
        orc.step(Xt, yt, ticks)
        spent += time.perf_counter() - t0
        done += 1
    return {"value": cfg.n * cfg.B * done / spent, "unit": "samples/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"first {done} iterations of the same workload, float64 numpy oracle "
                      f"(minibatch gather untimed), {spent:.1f} s"}


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="C3")
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
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="skip the per-launch HIP events (the roofline fields are then omitted)")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="for hardware-counter passes: three 256 MiB device copies (the calibration), "
                         "then five gradient launches of the workload; prints no bench line")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the DBW hot path here simulates all n workers on a single "
              f"MI355X; --gpus {args.gpus} is not supported.", file=sys.stderr)
        return 2

    import torch

    import paper_2004_14696_amd as dbw
    from dbw_inputs import get, init_params
    from dbw_inputs import generate as gen

    cfg = get(args.workload)
    if args.clock != cfg.clock:
        cfg = cfg.replace(clock=args.clock)
    if args.policy == "static" and not 1 <= args.k_static <= cfg.n:
        sys.exit(f"--policy static needs --k-static in [1, {cfg.n}]")
    cfg = cfg.replace(policy=args.policy, k_static=args.k_static if args.policy == "static" else 0,
                      estimator=args.estimator, g_rows=args.g_rows)
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    if args.traffic_probe:
        src = torch.full((64 * 1024 * 1024,), 1.0, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
    X, y = gen.dataset(cfg)
    Xd = torch.from_numpy(np.ascontiguousarray(X)).to(dev)
    yd = torch.from_numpy(np.ascontiguousarray(y)).to(dev)
    timing_pass = not args.no_kernel_timing
    total = args.warmup + args.steps * (2 if timing_pass else 1)
    rows = [torch.from_numpy(gen.batch_indices(cfg, t)).to(dev) for t in range(total)]
    ticks = [gen.round_trip_ticks(cfg, t) for t in range(total)]
    w = torch.from_numpy(init_params(cfg)).to(dev)
    ctx = dbw.Context(dbw.config_from(cfg, S=cfg.S))
    P = ctx.P

    if args.traffic_probe:
        G = torch.empty((cfg.n, P), dtype=torch.float32, device=dev)
        Lb = torch.empty(cfg.n, dtype=torch.float32, device=dev)
        for t in range(5):
            ctx.worker_grads(w, Xd, yd, rows=rows[t % len(rows)], G=G, loss=Lb)
        ctx.sync()
        print(f"traffic probe: 3 copies of 256 MiB, 5 gradient launches of {cfg.name}", flush=True)
        return 0

    ks = []
    for t in range(args.warmup):
        ks.append(ctx.step(w, Xd, yd, ticks[t], rows=rows[t], wait=False))
    ctx.sync()
    # timed region: host timers only (no device events in the launch stream)
    ctx.profile(2)
    ctx.profile_reset()
    stream = ctx.stream
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    t1 = args.warmup + args.steps
    for t in range(args.warmup, t1):
        ctx.step(w, Xd, yd, ticks[t], rows=rows[t], wait=False)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ctx.sync()
    gpu_ms = ev0.elapsed_time(ev1)
    host = {g: ctx.kernel_time(getattr(dbw.binding, "DBW_KT_" + g))
            for g in ("HOST_ESTIMATE", "HOST_STEP", "HOST_WAIT", "HOST_QUEUE")}
    # kernel-timing pass: the same loop continued with events around every
    # launch group (their cost stays out of the timed region above)
    grads_ms = grads_n = agg_ms = agg_n = choose_ms = choose_n = 0
    if timing_pass:
        ctx.profile(1)
        ctx.profile_reset()
        for t in range(t1, total):
            ctx.step(w, Xd, yd, ticks[t], rows=rows[t], wait=False)
        ctx.sync()
        agg_ms, agg_n = ctx.kernel_time(dbw.binding.DBW_KT_AGGREGATE)
        choose_ms, choose_n = ctx.kernel_time(dbw.binding.DBW_KT_CHOOSE)
        ctx.profile(False)
        # the gradient launch alone, back to back on the context stream with
        # the step's inputs, bracketed by two events (no per-launch events)
        G = torch.empty((cfg.n, P), dtype=torch.float32, device=dev)
        Lb = torch.empty(cfg.n, dtype=torch.float32, device=dev)
        ctx.worker_grads(w, Xd, yd, rows=rows[0], G=G, loss=Lb)
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for t in range(args.steps):
            ctx.worker_grads(w, Xd, yd, rows=rows[t1 + t], G=G, loss=Lb)
        g1.record(stream)
        torch.cuda.synchronize()
        grads_ms, grads_n = g0.elapsed_time(g1), args.steps
    ctx.profile(False)
    st = ctx.export_state()
    k_last = st["k_prev"]

    ms_per_step = wall * 1e3 / args.steps     # whole job: host estimate, launches, device work
    value = cfg.n * cfg.B / (ms_per_step / 1e3)
    gb = grads_bytes(cfg, P, True)
    grads_avg_s = grads_ms / max(grads_n, 1) / 1e3 if grads_n else float("nan")
    bound = roofline_bound(cfg)
    if bound == "hbm":
        achieved, peak, unit = gb / grads_avg_s / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved, peak, unit = grads_flops(cfg) / grads_avg_s / 1e12, MFMA_F32_PEAK_TFLOPS, "TFLOP/s"
    sb = step_bytes(cfg, P, k_last, True)
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
            "workload": f"{cfg.name}: softmax regression, n={cfg.n} workers x B={cfg.B} rows, d={cfg.d}, "
                        f"C={cfg.C}, minibatches gathered by index from a resident {cfg.S}x{cfg.d} dataset"
            if cfg.model == "softmax" else
            f"{cfg.name}: MLP {cfg.d}-{cfg.H}-{cfg.C}, n={cfg.n} workers x B={cfg.B} rows"
            if cfg.model == "mlp" else
            f"{cfg.name}: CNN 28x28 conv5x5(20)-pool-conv5x5(50)-pool-FC{cfg.H}-FC{cfg.C}, "
            f"n={cfg.n} workers x B={cfg.B} images gathered from a resident {cfg.S}-image dataset",
            "n": cfg.n, "B": cfg.B, "d": cfg.d, "C": cfg.C, "H": cfg.H, "P": P, "clock": cfg.clock,
            "policy": cfg.policy, "k_static": cfg.k_static, "estimator": cfg.estimator, "g_rows": cfg.g_rows,
        },
        "roofline": {
            "kernel": "worker gradients (dbw_worker_grads)",
            "bound": bound,
            "achieved": achieved,
            "peak": peak,
            "unit": unit,
            "frac": achieved / peak,
            "traffic": measured_traffic(cfg),
            "bytes_per_launch": gb,
            "flops_per_launch": grads_flops(cfg),
            "avg_launch_ms": grads_avg_s * 1e3,
            "launches": grads_n,
        },
        "step": {
            "gpu_ms_per_step": gpu_ms / args.steps,
            "wall_ms_per_step": wall * 1e3 / args.steps,
            "bytes_per_step": sb,
            "hbm_frac": sb / (ms_per_step / 1e3) / 1e9 / HBM_PEAK_GBS,
            "aggregate_and_stats_ms_per_step": agg_ms / args.steps if agg_n else None,
            "choose_ms_per_step": choose_ms / args.steps if choose_n else None,
            "host_estimate_ms_per_step": host["HOST_ESTIMATE"][0] / max(host["HOST_ESTIMATE"][1], 1),
            "host_step_call_ms": host["HOST_STEP"][0] / max(host["HOST_STEP"][1], 1),
            "host_wait_for_estimate_ms": host["HOST_WAIT"][0] / max(host["HOST_WAIT"][1], 1),
            "host_queue_ms": host["HOST_QUEUE"][0] / max(host["HOST_QUEUE"][1], 1),
            "k_last": k_last,
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, iters_cap=1000, budget_s=args.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
