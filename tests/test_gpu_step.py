"""GPU parity of a full DBW iteration (dbw_step) against the oracle.

Lockstep: before every iteration the oracle's state (parameters rounded to
fp32, estimator windows, arrival-time samples, clock) is imported into the
GPU context, one dbw_step runs, and every output is compared: the time
estimate, the objective and k (ties within 1e-6 relative accepted), the mask
(bit-exact), worker gradients and losses, the mean gradient, the statistics,
the parameter update, the smoothness estimate pushed into the state, and the
arrival-time grid and clock (exact).  Free-running: the GPU runs alone and
the oracle beside it; a GPU k that differs from the oracle's own choice must
be a near-tie of the oracle's objective, and the oracle then continues with
the GPU's k (masks, loss estimates and the final parameters compared)."""
import numpy as np
import pytest

from dbw_inputs import C1, C2, C3, C4, C5, C6, SOFTMAX, DBWConfig, TimeModel, gather, init_params
from dbw_inputs import generate as gen
from oracle import dbw as odbw
from oracle import model as omodel
from oracle import ps as ops
from gpu_util import (RTOL, cnn_best_flip, cnn_decision_flips, cnn_flip_deltas, host, k_acceptable,
                      mlp_best_flip, mlp_decision_flips, mlp_flip_deltas, rel_err, scalar_rel, to_dev)

torch = pytest.importorskip("torch")
pb = pytest.importorskip("paper_2004_14696_amd")

pytestmark = pytest.mark.gpu

EPS32 = float(np.finfo(np.float32).eps)

TINY = DBWConfig(name="tiny", model=SOFTMAX, n=6, B=16, d=40, C=4, S=500, iters=40, features="uniform",
                 labels="teacher", times=TimeModel(kind="shifted_exp", shift=0.5, rate=1.0), seed=4242)


def _setup(cfg):
    X, y = gen.dataset(cfg)
    ctx = pb.Context(pb.config_from(cfg, S=cfg.S))
    return X, y, ctx, to_dev(torch, X), to_dev(torch, y)


def _compare_iteration(cfg, rec, out, k_gpu, w_prev32, w_new, st_before, st_after, tag):
    n = cfg.n
    T_ref = rec["T_hat"]
    T_gpu = host(out["T_hat"])
    for kk in range(n):
        if T_ref[kk] is None:
            assert np.isnan(T_gpu[kk]), (tag, kk)
        else:
            assert T_gpu[kk] == pytest.approx(T_ref[kk], rel=1e-12), (tag, kk)
    assert k_acceptable(rec["objective"], k_gpu, rec["k"]), (tag, k_gpu, rec["k"])
    obj = host(out["objective"])
    if rec["objective"] is not None:
        for kk, v in enumerate(rec["objective"]):
            if v is not None:
                assert obj[kk] == pytest.approx(v, rel=1e-9, abs=1e-300), (tag, kk)
    Gg = host(out["G"])
    # with g_rows "selected" only the selected workers' rows are written, with
    # "none" no row is (the selected gradients are then checked through g, the
    # squared norms and the variance)
    if cfg.g_rows == "all":
        check_rows = range(n)
    elif cfg.g_rows == "selected":
        check_rows = rec["sel"] if k_gpu == rec["k"] else []
    else:
        check_rows = []
    for i in check_rows:
        assert rel_err(Gg[i], rec["G"][i]) <= RTOL, (tag, i)
    assert rel_err(host(out["loss"]), rec["loss"]) <= RTOL, tag
    if k_gpu != rec["k"]:
        return False           # a tie picked another k: the rest differs legitimately
    assert np.array_equal(host(out["mask"]), rec["mask"]), tag
    assert rel_err(host(out["g"]), rec["g"]) <= RTOL, tag
    s = host(out["stats"])
    k = rec["k"]
    assert scalar_rel(s[0], rec["gnorm2"]) <= RTOL, tag
    assert scalar_rel(s[1], rec["V_plus"]) <= RTOL, tag
    assert abs(s[2] - rec["N_plus"]) <= RTOL * max(rec["gnorm2"], rec["V_plus"] / k), tag
    assert scalar_rel(s[3], rec["F_hat"]) <= RTOL, tag
    sq = host(out["sqnorm"])
    ref_sq = np.zeros(n)
    for j in rec["sel"]:
        ref_sq[j] = float(rec["G"][j] @ rec["G"][j])
    assert rel_err(sq, ref_sq) <= RTOL, tag
    # parameter update: w_{t+1} - w_t = -eta g_t
    dw = w_new.astype(np.float64) - w_prev32.astype(np.float64)
    ref_dw = -cfg.eta * rec["g"]
    assert np.max(np.abs(dw - ref_dw)) <= RTOL * np.max(np.abs(ref_dw)) + 2 * EPS32 * np.max(np.abs(w_prev32)), tag
    # estimator state pushed by the GPU, from the GPU's own statistics
    assert st_after["t"] == st_before["t"] + 1 and st_after["k_prev"] == k, tag
    assert st_after["hV"][-1] == pytest.approx(s[1], rel=1e-15), tag
    assert st_after["hN"][-1] == pytest.approx(s[2], rel=1e-15, abs=1e-300), tag
    assert st_after["F_prev"] == pytest.approx(s[3], rel=1e-15), tag
    if rec["L_plus"] is None:
        assert st_after["hL"] == st_before["hL"], tag
    else:
        L_from_gpu_stats = odbw.l_estimate(cfg.eta, st_before["hN"][-1], st_before["hV"][-1], st_before["k_prev"],
                                           st_before["F_prev"], float(s[3]))
        assert st_after["hL"][:-1] == (st_before["hL"] + [None])[-cfg.D:][:-1], tag
        assert st_after["hL"][-1] == pytest.approx(L_from_gpu_stats, rel=1e-12), tag
    return True


def _seed_every_row(cfg, orc):
    """One fresh-start sample set in every row h (as if each k had been used
    once), from round-trip draws of iterations the run never reaches."""
    for h in range(1, cfg.n + 1):
        srt = sorted(int(x) for x in gen.round_trip_ticks(cfg, 10_000 + h))
        for i, v in enumerate(srt):
            orc.cnt[h - 1][i] += 1
            orc.tsum[h - 1][i] += v


def _lockstep(cfg, iters, seed_rows=False):
    X, y, ctx, Xd, yd = _setup(cfg)
    orc = odbw.DBWOracle(cfg, init_params(cfg))
    if seed_rows:
        _seed_every_row(cfg, orc)
    ties = 0
    for t in range(iters):
        idx = gen.batch_indices(cfg, t)
        ticks = gen.round_trip_ticks(cfg, t)
        w32 = orc.w.astype(np.float32)
        orc.w = w32.astype(np.float64)
        st = orc.export_state()
        ctx.import_state(st)
        ctx.import_samples(np.array(st["cnt"], np.int64), np.array(st["tsum"], np.int64), st["clock"])
        psw = cfg.clock == "psw"
        if psw:
            ctx.import_busy(np.array(orc.vclock.busy, np.int64))
        st_before = ctx.export_state()
        wd = to_dev(torch, w32)
        k_gpu = ctx.step(wd, Xd, yd, ticks, rows=to_dev(torch, idx), wait=True)
        out = ctx.step_outputs()
        ctx.sync()
        st_after = ctx.export_state()
        cnt_g, tsum_g, clock_g = ctx.export_samples()
        Xt, yt = gather(X, y, idx)
        if cfg.model == "mlp":
            w_at = orc.w.copy()
            _, _, A = omodel.mlp_worker_grads(w_at, Xt, yt, cfg.H, cfg.C, return_preact=True)
        elif cfg.model == "cnn":
            w_at = orc.w.copy()
            _, _, dec = omodel.cnn_worker_grads(w_at, Xt, yt, cfg.H, cfg.C, return_preact=True)
        V_window = odbw.window_mean(orc.hV, cfg.D)
        rec = orc.step(Xt, yt, ticks)
        # rows of G the GPU stored: every row, or (g_rows none on the paths
        # whose gradient kernels take the selection) those of its selection
        written = range(cfg.n) if cfg.g_rows == "all" else np.flatnonzero(host(out["mask"]))
        if cfg.model == "cnn":
            # pooling and ReLU choices within fp32 rounding may go either way:
            # each compared row's reference is the oracle with the subset of
            # those choices flipped that matches the GPU best (every parameter
            # block within RTOL), and the mean and the statistics are
            # recomputed from these references with the oracle's functions
            Gg = host(out["G"]).astype(np.float64)
            Gref = rec["G"].copy()
            for i in written:
                deltas = cnn_flip_deltas(w_at, Xt[i], yt[i], cfg.H, cfg.C, dec[i], cnn_decision_flips(dec[i]))
                err, Gref[i] = cnn_best_flip(Gg[i], rec["G"][i], deltas, cfg.H, cfg.C)
                assert err <= RTOL, (cfg.name, t, i, len(deltas))
            rec["G"] = Gref
            rec["g"] = ops.aggregate(Gref, rec["sel"])
            rec.update(ops.grad_stats(Gref, rec["sel"], rec["g"], rec["loss"],
                                      V_window if V_window is not None else 0.0))
        elif cfg.model == "mlp":
            # the same for the hidden ReLUs within rounding of zero
            Gg = host(out["G"]).astype(np.float64)
            Gref = rec["G"].copy()
            tau = 1e-6 * float(np.max(np.abs(A)))
            for i in written:
                flips = mlp_decision_flips(A[i], tau)
                assert len(flips) <= max(16, A[i].size // 2000), (cfg.name, t, i, len(flips))   # rare
                err, Gref[i] = mlp_best_flip(Gg[i], rec["G"][i],
                                             mlp_flip_deltas(w_at, Xt[i], yt[i], cfg.H, cfg.C, A[i], flips),
                                             cfg.d, cfg.H, cfg.C)
                assert err <= RTOL, (cfg.name, t, i, len(flips))
            rec["G"] = Gref
            rec["g"] = ops.aggregate(Gref, rec["sel"])
            rec.update(ops.grad_stats(Gref, rec["sel"], rec["g"], rec["loss"],
                                      V_window if V_window is not None else 0.0))
        same = _compare_iteration(cfg, rec, out, k_gpu, w32, host(wd), st_before, st_after, (cfg.name, t))
        ties += not same
        if iters >= 50:
            print(f"lockstep {cfg.name} g_rows={cfg.g_rows}: iteration {t} k={k_gpu}", flush=True)
        if same:
            assert np.array_equal(cnt_g, np.array(orc.cnt, np.int64)), (cfg.name, t)
            assert np.array_equal(tsum_g, np.array(orc.tsum, np.int64)), (cfg.name, t)
            assert clock_g == orc.clock, (cfg.name, t)
            if psw:
                assert np.array_equal(ctx.export_busy(), np.array(orc.vclock.busy, np.int64)), (cfg.name, t)
    assert ties <= max(1, iters // 20), f"{ties} near-tie choices in {iters} iterations"
    return orc


def test_lockstep_tiny_teacher():
    orc = _lockstep(TINY, TINY.iters)
    assert len(set(orc.ks)) > 1    # the teacher labels make k move


def test_lockstep_more_workers_than_inline_arguments():
    # 80 workers: the fused PS kernel reads T_hat and the arrival order from
    # pinned host memory (up to 64 they come in its kernel arguments)
    orc = _lockstep(TINY.replace(name="tiny80", n=80, iters=30), 30)
    assert len(set(orc.ks)) > 1


def test_lockstep_4_workers_full_run():
    _lockstep(C1, C1.iters)


def test_lockstep_16_workers_full_run():
    _lockstep(C2, C2.iters)


def test_lockstep_mlp_32_workers_full_run():
    _lockstep(C4, C4.iters)


def test_lockstep_push_and_wait_tiny():
    # Push & Wait: late workers finish their stale gradient first, and
    # workers still busy at a push skip it (censored samples)
    orc = _lockstep(TINY.replace(clock="psw"), TINY.iters)
    assert any(min(row) == 0 < max(row) for row in orc.cnt if max(row) > 0) or len(set(orc.ks)) > 1


def test_lockstep_push_and_wait_16_workers_slow_pair():
    # two workers five times slower: under Push & Wait they skip iterations
    cfg = C2.replace(clock="psw")
    orc = _lockstep(cfg, 60)
    censored = sum(1 for row in orc.cnt for a, b in zip(row, row[1:]) if b < a)
    assert censored > 0


def test_lockstep_static_k():
    orc = _lockstep(TINY.replace(policy="static", k_static=3), 20)
    assert orc.ks == [3] * 20


def test_lockstep_blind_dbw():
    # B-DBW: gain k, so k_t maximises k / T_hat_k
    orc = _lockstep(TINY.replace(policy="blind"), TINY.iters)
    assert orc.ks[:2] == [TINY.n] * 2 and len(set(orc.ks)) > 1


def test_lockstep_blind_dbw_push_interrupt_16_workers():
    orc = _lockstep(C2.replace(policy="blind", clock="psi"), 60)
    assert sum(map(sum, orc.cnt)) == sum(orc.ks)    # exactly k_t samples per iteration


def test_lockstep_naive_estimator():
    # the diagonal means of a grid seeded with one sample set per row, then
    # the run's own samples
    orc = _lockstep(TINY.replace(estimator="naive"), TINY.iters, seed_rows=True)
    assert len(set(orc.ks)) > 1


def test_lockstep_naive_estimator_push_and_wait_16_workers():
    _lockstep(C2.replace(estimator="naive", clock="psw"), 60, seed_rows=True)


def test_lockstep_push_interrupt_tiny():
    orc = _lockstep(TINY.replace(clock="psi"), TINY.iters)
    assert len(set(orc.ks)) > 1


def test_lockstep_cnn_small():
    # the MNIST-shaped CNN, 4 workers x 16 images, narrow first FC layer
    _lockstep(C6.replace(name="C6small", n=4, B=16, H=32, S=800, iters=10), 10)


def test_lockstep_cnn_workload_first_iteration():
    # 16 workers x 500 images, FC 800-500-10 (the oracle takes ~1 min)
    _lockstep(C6, 1)


def test_lockstep_64_workers_first_iterations():
    # every G row written and compared
    _lockstep(C3, 12)


def test_lockstep_64_workers_full_run_benchmarked_mode():
    # the mode the benchmark times: no G rows, the selected workers' slab
    # partials summed in the PS kernel; DBW reaches k = 1 on this workload
    orc = _lockstep(C3.replace(g_rows="none"), C3.iters)
    assert 1 in orc.ks and C3.n in orc.ks


def test_lockstep_256_workers_100_classes_first_iterations():
    _lockstep(C5, 3)


@pytest.mark.timeout(1500)
def test_lockstep_256_workers_100_classes_full_run_benchmarked_mode():
    # all 50 iterations of the largest workload in the benchmarked mode (the
    # matrix-core GEMM path writes every row; the PS reads the selected ones);
    # the oracle takes several seconds per iteration
    orc = _lockstep(C5.replace(g_rows="none"), C5.iters)
    assert len(set(orc.ks)) > 1


@pytest.mark.parametrize("base", [C2, C3], ids=lambda c: c.name)
@pytest.mark.parametrize("k", ["one", "all"])
def test_lockstep_benchmarked_mode_static_k(base, k):
    # the slab-source PS kernel at its extremes: a single selected worker (the
    # variance then takes the window mean) and every worker
    kk = 1 if k == "one" else base.n
    orc = _lockstep(base.replace(g_rows="none", policy="static", k_static=kk), 8)
    assert orc.ks == [kk] * 8


@pytest.mark.parametrize("cfg", [TINY, C1, C2.replace(name="C2psw", clock="psw", iters=80),
                                 C2.replace(name="C2psi_blind", clock="psi", policy="blind", iters=80)],
                         ids=lambda c: c.name)
def test_free_running_trajectory(cfg):
    X, y, ctx, Xd, yd = _setup(cfg)
    orc = odbw.DBWOracle(cfg, init_params(cfg))
    wd = to_dev(torch, init_params(cfg))
    forced = 0
    for t in range(cfg.iters):
        idx = gen.batch_indices(cfg, t)
        ticks = gen.round_trip_ticks(cfg, t)
        k_gpu = ctx.step(wd, Xd, yd, ticks, rows=to_dev(torch, idx), wait=True)
        Xt, yt = gather(X, y, idx)
        # the oracle's own choice from its own (drifted by fp32 rounding)
        # state; a different GPU k must be a near-tie of that objective, and
        # the oracle then continues with the GPU's k so that the rest of the
        # trajectory stays comparable
        T_hat = orc.time_estimate()
        k_orc, objective = orc.choose(T_hat)
        if k_gpu != k_orc:
            assert k_acceptable(objective, k_gpu, k_orc, tol=1e-4), (t, k_gpu, k_orc)
            forced += 1
        rec = orc.step(Xt, yt, ticks, T_hat=T_hat, k_force=k_gpu)
        out = ctx.step_outputs()
        assert np.array_equal(host(out["mask"]), rec["mask"]), t
        assert scalar_rel(host(out["stats"])[3], rec["F_hat"]) <= 1e-3, t
    assert forced <= max(1, cfg.iters // 20), forced
    assert rel_err(host(wd), orc.w) <= 1e-3


def test_lockstep_selected_rows_16_workers():
    # the selected workers' slab partials are aggregated in one kernel; only
    # their rows of G are written
    _lockstep(C2.replace(g_rows="selected"), 60)


def test_lockstep_selected_rows_64_workers_first_iterations():
    _lockstep(C3.replace(g_rows="selected"), 8)


@pytest.mark.parametrize("base", [C2, C3], ids=lambda c: c.name)
def test_slab_aggregation_matches_row_aggregation(base):
    # The same iterations with every row of G written and read back, with the
    # selected rows only, and with none: k, the mask, g, the update and the
    # losses are bitwise equal; the statistics differ only by the order of
    # their partial sums.  Rows of workers that were not selected keep stale
    # values in the fused modes.
    cfg = base.replace(policy="static", k_static=base.n // 2 + 1)
    X, y = gen.dataset(cfg)
    Xd, yd = to_dev(torch, X), to_dev(torch, y)
    modes = ("all", "selected", "none")
    ctxs = {m: pb.Context(pb.config_from(cfg.replace(g_rows=m), S=cfg.S)) for m in modes}
    ws = {m: to_dev(torch, init_params(cfg)) for m in modes}
    stale = 0
    for t in range(4):
        rows = to_dev(torch, gen.batch_indices(cfg, t))
        ticks = gen.round_trip_ticks(cfg, t)
        ks = {m: ctxs[m].step(ws[m], Xd, yd, ticks, rows=rows, wait=True) for m in modes}
        outs = {m: {k: host(v) for k, v in ctxs[m].step_outputs().items()} for m in modes}
        for m in modes:
            ctxs[m].sync()
        ref = outs["all"]
        assert ks["selected"] == ks["none"] == ks["all"] == cfg.k_static, t
        sel = np.flatnonzero(ref["mask"])
        for m in ("selected", "none"):
            o = outs[m]
            for name in ("mask", "g", "loss", "k", "b", "T_hat"):
                assert np.array_equal(o[name], ref[name], equal_nan=True), (m, t, name)
            assert np.array_equal(host(ws[m]), host(ws["all"])), (m, t)
            assert np.array_equal(o["stats"][3], ref["stats"][3]), (m, t)       # F_hat: same losses
            np.testing.assert_allclose(o["stats"], ref["stats"], rtol=1e-12, atol=0)
            np.testing.assert_allclose(o["sqnorm"], ref["sqnorm"], rtol=1e-5, atol=0)
        Gs, Ga = outs["selected"]["G"], ref["G"]
        assert np.array_equal(Gs[sel], Ga[sel]), t
        unsel = np.setdiff1d(np.arange(cfg.n), sel)
        stale += sum(not np.array_equal(Gs[j], Ga[j]) for j in unsel)
    assert stale > 0


def test_lockstep_mlp_selected_rows():
    # MLP with g_rows selected: the choice runs before the gradient kernels,
    # which store only the selected workers' G rows
    _lockstep(C4.replace(g_rows="selected"), 20)


@pytest.mark.parametrize("base", [
    C4,
    C5.replace(name="C5small", n=8, B=64, S=2000),
    C6.replace(name="C6small", n=4, B=16, S=800),
], ids=lambda c: c.name)
def test_skipped_rows_match_every_row(base):
    # Gradients from per-worker GEMM tiles: with g_rows selected the choice
    # and the selection run before the gradient kernels and only the
    # selected rows of G are stored.  k, the mask, g, the update, the losses
    # and the statistics are bitwise those of the run that stores every row;
    # the selected rows of G are equal; the others keep stale values.
    cfg = base.replace(policy="static", k_static=base.n // 2 + 1)
    X, y = gen.dataset(cfg)
    Xd, yd = to_dev(torch, X), to_dev(torch, y)
    modes = ("all", "selected")
    ctxs = {m: pb.Context(pb.config_from(cfg.replace(g_rows=m), S=cfg.S)) for m in modes}
    ws = {m: to_dev(torch, init_params(cfg)) for m in modes}
    stale = 0
    for t in range(3):
        rows = to_dev(torch, gen.batch_indices(cfg, t))
        ticks = gen.round_trip_ticks(cfg, t)
        ks = {m: ctxs[m].step(ws[m], Xd, yd, ticks, rows=rows, wait=True) for m in modes}
        outs = {m: {k: host(v) for k, v in ctxs[m].step_outputs().items()} for m in modes}
        for m in modes:
            ctxs[m].sync()
        ref, o = outs["all"], outs["selected"]
        assert ks["selected"] == ks["all"] == cfg.k_static, t
        for name in ("mask", "g", "loss", "k", "b", "T_hat", "stats", "sqnorm"):
            assert np.array_equal(o[name], ref[name], equal_nan=True), (t, name)
        assert np.array_equal(host(ws["selected"]), host(ws["all"])), t
        sel = np.flatnonzero(ref["mask"])
        assert np.array_equal(o["G"][sel], ref["G"][sel]), t
        unsel = np.setdiff1d(np.arange(cfg.n), sel)
        stale += sum(not np.array_equal(o["G"][j], ref["G"][j]) for j in unsel)
    assert stale > 0


def test_step_is_bitwise_deterministic():
    cfg = C2
    X, y = gen.dataset(cfg)
    res = []
    for _ in range(2):
        ctx = pb.Context(pb.config_from(cfg, S=cfg.S))
        Xd, yd = to_dev(torch, X), to_dev(torch, y)
        wd = to_dev(torch, init_params(cfg))
        ks = [ctx.step(wd, Xd, yd, gen.round_trip_ticks(cfg, t), rows=to_dev(torch, gen.batch_indices(cfg, t)),
                       wait=True) for t in range(6)]
        out = ctx.step_outputs()
        res.append((ks, host(wd), {k: host(v) for k, v in out.items()}))
    assert res[0][0] == res[1][0]
    assert np.array_equal(res[0][1], res[1][1])
    for name in res[0][2]:
        assert np.array_equal(res[0][2][name], res[1][2][name], equal_nan=True), name


def test_materialised_and_gathered_steps_agree():
    cfg = C1
    X, y = gen.dataset(cfg)
    ws = []
    for gathered in (True, False):
        ctx = pb.Context(pb.config_from(cfg, S=cfg.S if gathered else 0))
        wd = to_dev(torch, init_params(cfg))
        Xd, yd = (to_dev(torch, X), to_dev(torch, y)) if gathered else (None, None)
        for t in range(5):
            idx = gen.batch_indices(cfg, t)
            if gathered:
                ctx.step(wd, Xd, yd, gen.round_trip_ticks(cfg, t), rows=to_dev(torch, idx))
            else:
                Xt, yt = gather(X, y, idx)
                ctx.step(wd, to_dev(torch, Xt), to_dev(torch, yt), gen.round_trip_ticks(cfg, t))
        ctx.sync()
        ws.append(host(wd))
    assert np.array_equal(ws[0], ws[1])


def _exact_offset_batch(n, B, d, rng):
    """Minibatches whose worker gradients at W = 0 are exact in fp32 in any
    summation order, with a large common offset and a small spread across
    workers: features 1000 + m/16 (m < 16), every label 0, C = 4.  Then
    p = 1/4 exactly and G_i[j][c] = (1/B) sum_b x_bj (1/4 - [c = 0]): each
    product has at most 16 significant bits and a sum of B <= 256 of them at
    most 24."""
    X = (1000.0 + rng.integers(0, 16, size=(n, B, d)) / 16.0).astype(np.float32)
    y = np.zeros((n, B), np.int32)
    return X, y


@pytest.mark.parametrize("n,B,d,k", [
    (8, 16, 8, 2),         # one column tile: the choice and the aggregation in one kernel
    (8, 16, 8, 8),
    (6, 16, 40000, 2),     # P = 160000: separate choice, then the aggregation kernel
    (6, 16, 40000, 6),
    (4, 256, 64, 2),       # row slabs: the selected workers' slab partials summed in the PS kernel
    (4, 256, 64, 4),
])
def test_step_statistics_large_common_offset(n, B, d, k):
    # The PS kernels accumulate deviations from the fastest worker's row (a
    # shift that is itself a sample) and finish the variance from the shifted
    # sums.  Gradients of about -750 and 250 that differ across workers by
    # about 0.02: a sum of squares taken without the shift would lose every
    # digit of Eq. sumvariancekt in fp32.
    C = 4
    rng = np.random.default_rng(7000 + n * d + k)
    X, y = _exact_offset_batch(n, B, d, rng)
    ticks = rng.permutation(np.arange(1, n + 1, dtype=np.int64) * 1000)
    for g_rows in ("all", "none"):
        cfgc = pb.make_config("softmax", n, B, d, C, policy="static", k_static=k, g_rows=g_rows)
        ctx = pb.Context(cfgc)
        wd = to_dev(torch, np.zeros(d * C, np.float32))
        k_gpu = ctx.step(wd, to_dev(torch, X), to_dev(torch, y), ticks, wait=True)
        out = {name: host(v) for name, v in ctx.step_outputs().items()}
        ctx.sync()
        assert k_gpu == k
        Go, lo = omodel.softmax_worker_grads(np.zeros(d * C), X, y, C)
        sel, mask = ops.select_fastest(ticks, k)
        g = ops.aggregate(Go, sel)
        ref = ops.grad_stats(Go, sel, g, lo, 0.0)
        dev = Go[sel] - g[None, :]
        assert float(np.max(np.abs(dev))) < 1e-3 * float(np.max(np.abs(Go)))   # small spread
        assert np.array_equal(out["mask"], mask)
        assert rel_err(out["g"], g) <= 1e-6, g_rows
        st = out["stats"]
        assert scalar_rel(st[1], ref["V_plus"]) <= RTOL, (g_rows, st[1], ref["V_plus"])
        assert scalar_rel(st[0], ref["gnorm2"]) <= RTOL, g_rows
        assert abs(st[2] - ref["N_plus"]) <= RTOL * max(ref["gnorm2"], ref["V_plus"] / k), g_rows
        assert rel_err(out["sqnorm"], ref["sqnorm"]) <= RTOL, g_rows
        assert rel_err(host(wd), -0.1 * g) <= 1e-6, g_rows
