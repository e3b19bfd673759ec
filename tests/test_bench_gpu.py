"""The benchmark's output: one JSON line with the fields its readers rely on
(the throughput and its timing statistics, the roofline of the dominant
kernel, the oracle's CPU baseline and the parity of the timed outputs
against it), here on the small workload with a short oracle sample, and
each order's line with its own metric."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    print(f"case bench {' '.join(args)}", flush=True)
    r = subprocess.run([sys.executable, "-u", "bench.py", *args], cwd=ROOT, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, r.stdout[-3000:]
    return json.loads(lines[0])


def test_bench_line_fields_and_parity():
    d = _bench("--workload", "tiny", "--steps", "4", "--warmup", "2", "--cpu-steps", "512")
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline", "parity",
                "lane_steps_g_per_s", "ms_per_step_stats", "kernels", "vram"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 4 and d["warmup"] == 2
    assert d["higher_is_better"] is True and d["vs_baseline"] is None and d["dtype"] == "f32"
    cfg = d["config"]
    assert cfg["workload"] == "tiny" and "model" not in cfg
    B, L, D, N = cfg["batch"], cfg["seq_len"], cfg["d_inner"], cfg["d_state"]
    ms = d["ms_per_step"]
    assert ms > 0 and d["ms_per_step_stats"]["min"] <= ms <= d["ms_per_step_stats"]["max"]
    assert d["value"] == pytest.approx(B * L * D / (ms * 1e-3) / 1e9, rel=2e-3, abs=1e-3)   # 3 decimals
    assert d["lane_steps_g_per_s"] == pytest.approx(B * L * D * N / (ms * 1e-3) / 1e9, rel=2e-3, abs=0.06)
    rf = d["roofline"]
    assert rf["bound"] in ("hbm", "mfma", "alu") and rf["unit"] in ("GB/s", "TFLOP/s")
    assert rf["peak"] > 0 and rf["achieved"] > 0
    assert rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-2, abs=1e-4)
    assert rf["peak_unpacked"] == pytest.approx(78.64, abs=0.01) and rf["frac_unpacked"] >= rf["frac"]
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["sample"]
    assert cb["lane_steps_g_per_s"] == pytest.approx(cb["value"] * N, rel=1e-3, abs=2e-6)
    par = d["parity"]
    assert par["y_rel_l2"] <= 1e-5 and par["dy_rel_l2"] <= 1e-5, par
    assert par["channels"] == D and 0 < par["steps"] <= L
    assert par["tail_dy_rel_l2"] <= 1e-5, par


@pytest.mark.parametrize("order", [2, 3])
def test_bench_line_of_each_order(order):
    d = _bench("--workload", "tiny", "--order", str(order), "--steps", "3", "--warmup", "1", "--no-cpu")
    assert d["value"] > 0 and d["cpu_baseline"] is None
    assert d["roofline"]["bound"] == "alu" and d["roofline"]["frac"] > 0
    assert d["config"]["workload"].startswith("tiny")
