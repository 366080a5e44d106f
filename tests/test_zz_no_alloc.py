"""dbw_grad_stats_static, the statistics call for callers that cannot
allocate: its scratch is the library's static device array.  Checked through
the C ABI against the context call dbw_grad_stats (the same kernels, so the
results must be bitwise equal), on two calls in a row with a smaller input
the second time, and its argument checks on the host."""
import ctypes

import numpy as np
import pytest

from gpu_util import RTOL, host, rel_err, scalar_rel, to_dev
from oracle import ps as ops

pb = pytest.importorskip("paper_2004_14696_amd.binding")


def _inputs(rng, n, P, k, offset=0.05):
    G = (rng.standard_normal((n, P)) * 0.3 + offset).astype(np.float32)
    loss = rng.uniform(1.0, 3.0, size=n).astype(np.float32)
    sel = sorted(rng.choice(n, size=k, replace=False).tolist())
    mask = np.zeros(n, np.uint8)
    mask[sel] = 1
    g = ops.aggregate(G, sel).astype(np.float32)
    return G, loss, mask, sel, g


def _ctx_for_P(n, P):
    C = next(c for c in range(2, 4097) if P % c == 0)
    return pb.Context(pb.make_config("softmax", n, 1, P // C, C))


@pytest.mark.gpu
def test_static_stats_match_the_context_call_twice_second_smaller():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2024)
    for n, P, k in ((64, 30720, 40), (16, 7840, 5)):
        G, loss, mask, sel, g = _inputs(rng, n, P, k)
        Gd, md, gd, ld = to_dev(torch, G), to_dev(torch, mask), to_dev(torch, g), to_dev(torch, loss)
        sq_s, st_s = pb.grad_stats_static(Gd, md, k, gd, ld)
        ctx = _ctx_for_P(n, P)
        sq_c, st_c = ctx.grad_stats(Gd, md, k, gd, ld)
        ctx.sync()
        torch.cuda.synchronize()
        assert torch.equal(sq_s, sq_c), (n, P)
        assert torch.equal(st_s, st_c), (n, P, host(st_s), host(st_c))
        ref = ops.grad_stats(G, sel, g.astype(np.float64), loss)
        st = host(st_s)
        assert rel_err(host(sq_s), ref["sqnorm"]) <= RTOL
        assert scalar_rel(st[0], ref["gnorm2"]) <= RTOL
        assert scalar_rel(st[1], ref["V_plus"]) <= RTOL
        assert scalar_rel(st[3], ref["F_hat"]) <= RTOL


@pytest.mark.gpu
def test_static_stats_k1_window_and_bad_masks():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    n, P = 5, 640
    G, loss, mask, sel, g = _inputs(rng, n, P, 1)
    Gd, md, gd, ld = to_dev(torch, G), to_dev(torch, mask), to_dev(torch, g), to_dev(torch, loss)
    hV = [2.0, 4.0, 9.0]
    ctx = _ctx_for_P(n, P)
    ctx.import_state({"t": 3, "k_prev": 5, "hV": hV, "hN": [0.1, 0.2, 0.3], "hL": [1.0, 2.0], "nF": 2,
                      "F_prev": 1.0, "F_prev2": 1.1})
    sq_c, st_c = ctx.grad_stats(Gd, md, 1, gd, ld)
    sq_s, st_s = pb.grad_stats_static(Gd, md, 1, gd, ld, V_window=float(np.mean(hV)))
    ctx.sync()
    torch.cuda.synchronize()
    assert torch.equal(sq_s, sq_c) and torch.equal(st_s, st_c)
    # a mask with more or fewer ones than k: NaN statistics (no flag to raise)
    for k in (2, 1):
        bad = mask.copy() if k == 2 else np.ones(n, np.uint8)
        _, st = pb.grad_stats_static(Gd, to_dev(torch, bad), k, gd, ld)
        torch.cuda.synchronize()
        assert np.all(np.isnan(host(st))), k
    # and the next good call is unaffected
    _, st = pb.grad_stats_static(Gd, md, 1, gd, ld, V_window=float(np.mean(hV)))
    torch.cuda.synchronize()
    assert torch.equal(st, st_c)


def test_static_stats_argument_checks_on_the_host():
    # rejected before any HIP call
    lib = pb.load_library()
    p = ctypes.c_void_p(256)
    null = ctypes.c_void_p(0)
    stream = ctypes.c_void_p(0)

    def call(n, P, k, ptr=p, V=0.0):
        return lib.dbw_grad_stats_static(n, P, ptr, p, k, p, p, V, p, p, stream)

    assert call(0, 64, 1) == pb.DBW_EINVAL
    assert call(pb.DBW_MAX_N + 1, 64, 1) == pb.DBW_EINVAL
    assert call(4, 0, 1) == pb.DBW_EINVAL
    assert call(4, 64, 1, ptr=null) == pb.DBW_EINVAL
    assert call(4, 64, 0) == pb.DBW_ERANGE
    assert call(4, 64, 5) == pb.DBW_ERANGE
    assert call(4, 64, 2, V=float("nan")) == pb.DBW_EINVAL
    # 1024 rows x 8192 column tiles of partial norms: 32 MiB of scratch
    assert call(1024, 8192 * 256, 3) == pb.DBW_EUNSUPPORTED
    assert b"scratch" in lib.dbw_last_error(None)
    assert call(4, (1 << 29) + 1, 2) == pb.DBW_EUNSUPPORTED
