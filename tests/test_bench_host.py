"""bench.py's host-side parts, on the CPU: the one-GPU refusal, the paper-order flop
count, the algorithmic byte models, the HBM-traffic gate on the committed
profiles, the CPU baseline record and the sub-record of each workload."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2310_12298_amd.workloads import CONFIGS  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120, cwd=ROOT)
    assert res.returncode == 2
    assert "exactly one GPU" in res.stderr and res.stdout == ""


def test_paper_order_flops_count_each_product_once():
    # Per factor of size d with statistic rank k: A^2 and A^4 (symmetric: d^3 each), X, X X and
    # A P (2 d^3 each), the Gram product (symmetric: d^2 k); plus L G (2 m^2 n) and (L G) R (2 m n^2).
    def by_parts(m, n):
        factor = lambda d, k: 2 * d ** 3 + 3 * 2 * d ** 3 + d * d * k
        return factor(m, n) + factor(n, m) + 2 * m * m * n + 2 * m * n * n
    for m, n in [(1, 1), (64, 576), (512, 4608), (7, 3)]:
        assert bench.falg_paper(m, n) == by_parts(m, n)


def test_byte_models():
    shapes = [(3, 5), (64, 576)]
    mn = 3 * 5 + 64 * 576
    assert bench.stage_bytes(shapes) == {"weight": 12 * mn, "stage_in": 20 * mn}
    fac = 3 * 3 + 5 * 5 + 64 * 64 + 576 * 576
    assert bench.step_bytes(shapes, True) == 4 * (7 * mn + 2 * fac)
    assert bench.step_bytes(shapes, False) == 4 * (7 * mn + fac)


def test_traffic_is_read_only_for_the_sources_it_was_measured_with(monkeypatch):
    for config in CONFIGS:
        path = bench.profile_path(config)
        assert os.path.exists(path), f"{path}: every workload has a committed profile"
        v = bench.measured_traffic(config)
        assert v is None or v > 0
    monkeypatch.setattr(bench, "kernel_sources_sha256", lambda: "0" * 64)
    assert all(bench.measured_traffic(c) is None for c in CONFIGS)


def test_cpu_baseline_record():
    shapes, sigma, _ = CONFIGS["single_64x576"]
    rec = dict(bench.cpu_baseline(shapes, sigma, 0, 0.2), **bench.cpu_info())
    assert rec["kind"] == "oracle" and rec["unit"] == "steps/s"
    assert rec["value"] > 0 and rec["cores"] >= 1 and rec["os_cpu_count"] == os.cpu_count()
    assert "fp64 oracle steps 1.." in rec["sample"]
    json.dumps(rec)


def test_workload_sub_record_fields():
    res = {"config": "many_small", "steps": 200, "value": 1500.0, "ms_per_step": 0.66,
           "gemm": {"achieved": 60.0}, "step_roofline": {"frac": 0.33, "bound": "mfma"},
           "forms": {"explicit": 811, "factored": 132, "squared": 81},
           "hbm": {"weight": {"frac": 0.8}, "stage_in": {"frac": 0.85}}}
    rec = bench.summary(res)
    assert rec["gemm_frac"] == pytest.approx(60.0 / 157.3)
    assert rec["workload"] == bench.WORKLOAD_NAMES["many_small"] and rec["unit"] == "steps/s"
    assert set(rec["hbm_frac"]) == {"weight", "stage_in"}
    json.dumps(rec)


def test_layers_option_parses_shape_lists():
    assert bench.parse_layers("128x128*3,64x576") == [(128, 128)] * 3 + [(64, 576)]
    assert bench.parse_layers(" 1x1 ") == [(1, 1)]
    for bad in ("128", "0x4", "4x4*0", "axb", "4x4*z"):
        with pytest.raises(SystemExit):
            bench.parse_layers(bad)
