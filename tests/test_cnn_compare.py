"""The CNN comparison helpers of the GPU tests, checked on the oracle alone
(no GPU): a result with any subset of the within-rounding choices taken the
other way is accepted, a perturbation of any parameter block is not."""
import numpy as np

from oracle import model as omodel
from gpu_util import RTOL, cnn_best_flip_err, cnn_blocks, cnn_decision_flips, cnn_flip_deltas


def _case():
    rng = np.random.default_rng(66)
    B, H, C = 3, 8, 4
    X = rng.random((B, 784)) * (rng.random((B, 784)) > 0.5)
    y = rng.integers(0, C, size=B)
    w = rng.uniform(-0.15, 0.15, size=omodel.cnn_param_count(H, C))
    G, _, dec = omodel.cnn_worker_grads(w, X[None], y[None], H, C, return_preact=True)
    return w, X, y, H, C, G[0], dec[0]


def test_flips_are_found_and_each_one_is_accepted_either_way():
    w, X, y, H, C, G, dec = _case()
    # loose thresholds so that this small case has choices to flip
    flips = cnn_decision_flips(dec, frac=2e-2, conv_frac=2e-3)
    keys = {f[1] for f in flips}
    assert {"code1", "code2", "on1", "on2"} <= keys, keys
    deltas = cnn_flip_deltas(w, X, y, H, C, dec, flips)[:6]
    assert len(deltas) >= 3
    assert cnn_best_flip_err(G, G, deltas, H, C) == 0.0
    for m in (1, 5, (1 << len(deltas)) - 1):
        flipped = G + sum(d for i, d in enumerate(deltas) if m >> i & 1)
        assert cnn_best_flip_err(flipped, G, deltas, H, C) <= 1e-12


def test_flip_delta_is_the_oracle_with_that_choice_changed():
    w, X, y, H, C, G, dec = _case()
    flips = cnn_decision_flips(dec, frac=2e-2, conv_frac=2e-3)
    b, key, idx, val = next(f for f in flips if f[1] == "code2")
    d = cnn_flip_deltas(w, X, y, H, C, dec, [(b, key, idx, val)])
    # the whole worker run with the same change gives the same gradient
    P1, c1 = omodel.maxpool2(dec["Z1"])
    P2, c2 = omodel.maxpool2(dec["Z2"])
    own = {"code1": c1, "on1": P1 > 0, "code2": c2.copy(), "on2": P2 > 0, "on3": dec["A3"] > 0}
    own["code2"][(b, *idx)] = val
    Gf = omodel.cnn_worker_grads(w, X[None], y[None], H, C, decisions=own)[0][0]
    assert len(d) == 1
    np.testing.assert_allclose(G + d[0], Gf, rtol=0, atol=1e-12 * np.abs(G).max())


def test_a_perturbed_block_is_rejected():
    w, X, y, H, C, G, dec = _case()
    deltas = cnn_flip_deltas(w, X, y, H, C, dec, cnn_decision_flips(dec))
    for lo, hi in cnn_blocks(H, C):
        a = G.copy()
        j = lo + int(np.argmax(np.abs(G[lo:hi])))
        a[j] += 3 * RTOL * np.abs(G[lo:hi]).max()
        assert cnn_best_flip_err(a, G, deltas, H, C) > RTOL, (lo, hi)
