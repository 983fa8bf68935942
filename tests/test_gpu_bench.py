"""bench.py's output contract on the GPU: one JSON line with the metric, the roofline of the dominant kernel
(measured on its launch stream) and the bandwidth steps, from a short run of the benchmark workload."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line():
    print("[bench] short run of bench.py", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--steps", "3", "--warmup", "3",
                        "--min-warmup-seconds", "0.2", "--no-cpu-baseline", "--workload",
                        "bf16_T4096_d1024_f2816_E16_k2"], capture_output=True, text=True, timeout=110)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    out = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
                "vs_baseline", "dtype", "data", "config", "roofline"):
        assert key in out, key
    assert out["n_gpus"] == 1 and out["steps"] == 3 and out["warmup"] == 3 and out["warmup_steps_run"] >= 3
    assert out["value"] > 0 and out["ms_per_step"] > 0 and out["dtype"] == "bf16"
    assert out["config"]["workload"] == "bf16_T4096_d1024_f2816_E16_k2"
    roof = out["roofline"]
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s" and roof["peak"] == 2516.6
    assert 0 < roof["frac"] < 1 and abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    assert set(out["hbm_steps_warmup"]) >= {"route_fwd", "permute", "combine", "combine_bwd", "unpermute"}


def test_bench_dense_reference_line():
    """bench.py --dense-reference: one JSON line with the vendor GEMM's rate on the workload's three expert shapes."""
    print("[bench] dense reference", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--dense-reference", "--workload",
                        "bf16_T4096_d1024_f2816_E16_k2"], capture_output=True, text=True, timeout=110)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    out = json.loads(lines[0])
    assert out["workload"] == "bf16_T4096_d1024_f2816_E16_k2"
    assert set(out["shapes"]) == {"gate_up", "down", "dx"}
    rows = 4096 * 2
    assert (out["shapes"]["gate_up"]["M"], out["shapes"]["gate_up"]["K"], out["shapes"]["gate_up"]["N"]) == (rows, 1024, 5632)
    for s in out["shapes"].values():
        assert s["us"] > 0 and 0 < s["frac"] < 1 and abs(s["TFLOP/s"] / 2516.6 - s["frac"]) < 1e-3
