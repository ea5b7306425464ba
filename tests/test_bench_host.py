"""Host-side logic of bench.py (CPU only): the algorithmic byte counts behind
`value` and `roofline`, the median and bootstrap interval, the counter-CSV
summaries behind `profiles/`, and the refusal of more than one GPU."""

import csv
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_21137_amd.configs import (NEMOTRON3_B1, QWEN3_B1, QWEN3_B16,  # noqa: E402
                                          WIDE_SKEW_B4)


def test_compressed_bytes_qwen3_by_hand():
    # per active expert: gate and up codes H*I/d each, V_gate and V_up r*I bf16,
    # down codes I*H/d and A_e I*r bf16 (Qwen3 shape: 2048, 768, d=8, r=128)
    per = 2 * (2048 * 768 // 8) + 2 * (128 * 768 * 2) + (768 * 2048 // 8) + (768 * 128 * 2)
    assert per == 1_179_648
    b = bench.compressed_bytes(QWEN3_B1, 8)
    assert b["per_expert_gateup"] + b["per_expert_down"] == per
    # shared per launch: B (r*H bf16) and three code books (K*d bf16 each);
    # U belongs to the routing kernel's z items
    shared_expert = 128 * 2048 * 2 + 3 * 256 * 8 * 2
    assert shared_expert == 536_576
    assert b["expert_kernel"] == 8 * per + shared_expert == 9_973_760
    assert b["compressed"] == b["expert_kernel"] + 2048 * 128 * 2
    assert b["route_kernel"] == 2048 * 128 * 2 + 128 * 4 + 2048 * 128 * 2
    # separate gate and up bases double U
    assert bench.compressed_bytes(QWEN3_B16, 80, z_sep=True)["compressed"] == \
        bench.compressed_bytes(QWEN3_B16, 80)["compressed"] + 2048 * 128 * 2


def test_compressed_bytes_up_only_has_no_gate():
    w = NEMOTRON3_B1
    b = bench.compressed_bytes(w, 1)
    assert b["per_expert_gateup"] == w.H * w.I // w.d + w.r * w.I * 2
    assert b["expert_kernel"] - b["per_expert_gateup"] - b["per_expert_down"] == \
        w.r * w.H * 2 + 2 * w.K * w.d * 2  # B and the up and down books


def test_dense_bytes():
    w = QWEN3_B1
    d = bench.dense_bytes(w, 8, "dense")
    assert d["expert_kernel"] == 8 * 3 * 2048 * 768 * 2 == 75_497_472
    dd = bench.dense_bytes(w, 8, "dense_down")
    gu = 2 * (2048 * 768 // 8) + 2 * (128 * 768 * 2)
    assert dd["expert_kernel"] == 8 * (gu + 768 * 2048 * 2) + 2 * 256 * 8 * 2
    assert dd["weights"] == dd["expert_kernel"] + 2048 * 128 * 2
    # the wide layer at its own shape
    assert bench.dense_bytes(WIDE_SKEW_B4, 6, "dense")["weights"] == 6 * 3 * 4096 * 1536 * 2


def test_bootstrap_ci():
    rng = np.random.default_rng(3)
    v = 25.0 + rng.standard_normal(200)
    med, lo, hi = bench.bootstrap_ci(v)
    assert med == pytest.approx(float(np.median(v)))
    assert lo <= med <= hi
    assert hi - lo < 0.6  # ~3.9 standard errors of a median of 200 unit normals
    assert bench.bootstrap_ci(v) == (med, lo, hi)  # seeded: the same interval every run
    c = bench.bootstrap_ci([7.0] * 30)
    assert c == (7.0, 7.0, 7.0)


def _write_csv(path, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for r in rows:
            wr.writerow(dict(zip(("Kernel_Name", "Counter_Name", "Counter_Value"), r)))


def test_summarize_counters(tmp_path, capsys):
    ke, kr = "void cardan::k_expert<8, 1, 0>(...)", "cardan::k_route(...)"
    p = tmp_path / "c.csv"
    _write_csv(p, [(ke, "SQ_INSTS_LDS", 10), (ke, "SQ_INSTS_LDS", 20), (ke, "GRBM_GUI_ACTIVE", 5),
                   (kr, "SQ_INSTS_LDS", 4), ("__amd_rocclr_copyBuffer", "SQ_INSTS_LDS", 99)])
    bench.summarize_counters([str(p)])
    out = json.loads(capsys.readouterr().out)
    assert out["kernel_source_hash"] == bench.kernel_source_hash()
    m = out["per_dispatch_mean"]
    assert set(m) == {ke, kr}  # only the library's kernels
    assert m[ke]["SQ_INSTS_LDS"] == 15.0 and m[ke]["GRBM_GUI_ACTIVE"] == 5.0
    assert m[kr]["SQ_INSTS_LDS"] == 4.0


def test_summarize_pmc_scales_by_the_copy(tmp_path, monkeypatch):
    ke = "void cardan::k_expert<8, 2, 0>(...)"
    copy = "__amd_rocclr_copyBuffer"
    f, w, cf, cw = (tmp_path / n for n in ("f.csv", "w.csv", "cf.csv", "cw.csv"))
    _write_csv(f, [(ke, "FETCH_SIZE", 1000.0), (ke, "FETCH_SIZE", 3000.0)])
    _write_csv(w, [(ke, "WRITE_SIZE", 100.0)])
    # a 1 MiB copy whose counters read half (fetch) and all (write) of it
    _write_csv(cf, [(copy, "FETCH_SIZE", 512.0)])
    _write_csv(cw, [(copy, "WRITE_SIZE", 1024.0)])
    out_dir = tmp_path / "profiles"
    out_dir.mkdir()
    src_hash = bench.kernel_source_hash()
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: src_hash)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))  # the record goes to <ROOT>/profiles

    class Args:
        summarize_pmc = [str(f), str(w), str(cf), str(cw)]
        calibrate_copy_mb = 1
        pmc_kernel = "k_expert"
        pmc_name = "wl"
        workload = "wl"

    bench.summarize_pmc(Args)
    rec = json.load(open(out_dir / "k_expert_wl_pmc.json"))
    assert rec["copy_calibration"]["fetch_scale"] == pytest.approx(2.0)
    assert rec["copy_calibration"]["write_scale"] == pytest.approx(1.0)
    assert rec["hbm_read_bytes_per_launch"] == 2000 * 1024 * 2
    assert rec["hbm_write_bytes_per_launch"] == 100 * 1024
    assert rec["hbm_bytes_per_launch"] == rec["hbm_read_bytes_per_launch"] + rec["hbm_write_bytes_per_launch"]


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
