"""Host-side pieces of bench.py: the algorithmic byte and flop counts behind
the roofline, the choice of bound, the guard on committed counter summaries,
and the single-GPU contract."""
import hashlib
import json

import pytest

import bench
from dbw_inputs import get


def test_grads_bytes_softmax_default_workload():
    # 64 x 256 gathered rows of 3072 floats, their labels and row indices, the
    # 3072 x 10 parameters once, 64 gradient rows and losses
    cfg = get("C3")
    P = cfg.d * cfg.C
    rows = cfg.n * cfg.B
    expect = 4 * (rows * cfg.d + 2 * rows + P + cfg.n * P + cfg.n)
    assert bench.grads_bytes(cfg, P, True) == expect == 209445120


def test_grads_flops_and_bound():
    c3, c4, c5 = get("C3"), get("C4"), get("C5")
    assert bench.grads_flops(c3) == 4.0 * 64 * 256 * 3072 * 10
    assert bench.grads_flops(c4) == 4.0 * 32 * 64 * 784 * 512 + 6.0 * 32 * 64 * 512 * 10
    assert bench.roofline_bound(c3) == "hbm"
    assert bench.roofline_bound(c4) == "mfma"
    assert bench.roofline_bound(c5) == "mfma"


def _summary(tmp_path, src_rel, digest, value):
    rec = {"kernel_sources_sha256": {src_rel: digest}, "traffic_bytes_per_launch": value}
    p = tmp_path / "traffic.md"
    p.write_text("# traffic\n\nmachine-readable: " + json.dumps(rec) + "\n")
    return str(p)


def test_measured_traffic_follows_kernel_source(tmp_path, monkeypatch):
    src_rel = "paper_2004_14696_amd/csrc/k_softmax.hip"
    digest = hashlib.sha256(open(src_rel, "rb").read()).hexdigest()
    cfg = get("C3")
    monkeypatch.setitem(bench.TRAFFIC_FILE, "C3", _summary(tmp_path, src_rel, digest, 123))
    assert bench.measured_traffic(cfg) == 123
    # a summary taken on another version of the kernel is not used
    monkeypatch.setitem(bench.TRAFFIC_FILE, "C3", _summary(tmp_path, src_rel, "0" * 64, 123))
    assert bench.measured_traffic(cfg) is None


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err


def test_roofline_block_warm_and_cold():
    # C5: 1.61e11 useful flops per launch; 2 ms warm and 2.5 ms cold
    cfg = get("C5")
    r = bench.roofline_block(cfg, cfg.d * cfg.C, 2.0, 2.5, 20)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert r["achieved"] == pytest.approx(bench.grads_flops(cfg) / 2e-3 / 1e12)
    assert r["frac"] == pytest.approx(r["achieved"] / bench.MFMA_F32_PEAK_TFLOPS)
    assert r["cold"]["achieved"] == pytest.approx(r["achieved"] * 2.0 / 2.5)
    c3 = get("C3")
    r3 = bench.roofline_block(c3, c3.d * c3.C, 0.05, 0.06, 20)
    assert r3["bound"] == "hbm" and r3["unit"] == "GB/s"
    assert r3["achieved"] == pytest.approx(209445120 / 0.05e-3 / 1e9)
