"""Host-side checks of bench.py: its refusal of more than one GPU, the algorithmic FLOP and byte counts it
reports against, the traffic record lookup and the workload names (no GPU is touched here)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2506_02965_amd.synth import CONFIGS, LayerConfig  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_layer_flops_by_hand():
    cfg = LayerConfig("f", T=10, d=4, f=6, E=3, k=2, n_shared=1)
    rows = 20 + 10                                     # routed rows + one shared expert on every token
    fwd = 6 * 4 * 6 * rows + 2 * 10 * 4 * 3            # SwiGLU expert 6df per row, router 2TdE
    bwd = 12 * 4 * 6 * rows + 4 * 10 * 4 * 3           # 12df per row, router adjoint 4TdE
    assert bench.layer_flops(cfg, 20, backward=False) == fwd
    assert bench.layer_flops(cfg, 20) == fwd + bwd
    no_router = LayerConfig("g", T=10, d=4, f=6, E=3, k=2, n_shared=1, router_backward=False)
    assert bench.layer_flops(no_router, 20) == fwd + 12 * 4 * 6 * rows


def test_hbm_step_bytes_by_hand():
    cfg = LayerConfig("b", T=8, d=16, f=32, E=4, k=2, n_shared=1)   # bf16: 2 bytes per element
    kernels = {n: {"avg_us": 1.0} for n in ("route_fwd", "permute_hist", "permute_scatter", "permute_gather",
                                            "combine", "combine_bwd", "unpermute")}
    out = bench.hbm_steps(cfg, 16, kernels)
    row = 16 * 2                                         # one d-row in bytes
    assert out["route_fwd"]["bytes"] == 8 * row + 4 * row + 4 * 8 * 4 + 8 * 8 * 2
    assert out["permute"]["bytes"] == 8 * row + 16 * row + 8 * 8 * 2
    assert out["permute"]["us"] == 3.0                   # three launches (histogram, scatter, gather)
    assert out["combine"]["bytes"] == 16 * row + 8 * row + 8 * row + 8 * 8 * 2
    assert out["combine_bwd"]["bytes"] == 8 * row + 2 * 16 * row + 8 * 8 * 2
    assert out["unpermute"]["bytes"] == 16 * row + 8 * row + 8 * row + 4 * 8 * 2


def test_traffic_record_matches_only_its_kernel_workload_and_sources():
    rec = {}
    for line in open(bench.TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            rec[k.strip()] = v.strip()
    assert bench.measured_traffic(rec["kernel"], "another_workload") is None
    assert bench.measured_traffic("another_kernel", rec["workload"]) is None
    got = bench.measured_traffic(rec["kernel"], rec["workload"])
    if rec["gemm_sources"] != bench.gemm_source_digest():
        assert got is None                               # stale record: the GEMM sources changed since
    else:
        cal = bench.COPY_CAL_BYTES / 1024
        want = (float(rec["fetch_kib_per_launch"]) * cal / float(rec["copy_fetch_kib"])
                + float(rec["write_kib_per_launch"]) * cal / float(rec["copy_write_kib"])) * 1024
        assert got == round(want)


def test_workloads_by_name_and_position():
    for i, c in CONFIGS.items():
        assert bench.pick_workload(c.name) is c
        assert bench.pick_workload(str(i)) is c
    with pytest.raises(SystemExit):
        bench.pick_workload("no_such_workload")


def test_default_workload_is_the_largest():
    """The headline runs on the layer with the most work per step (T=8192, d=4096, f=14336, E=8, top-2)."""
    big = max(CONFIGS.values(), key=lambda c: c.T * c.k * c.d * c.f)
    assert bench.DEFAULT_WORKLOAD == big.name == CONFIGS[4].name


def test_host_info_fields():
    info = bench.host_info()
    assert info["cores_available"] == len(os.sched_getaffinity(0))
    assert info["blas_threads"] >= 1 and isinstance(info["cpu_model"], str) and info["blas"]


def test_cpu_baseline_sample_is_bounded():
    """The oracle baseline on a small layer: routing of every token plus whole experts, stopping once the
    time bound is met (here at once: one expert), with the FLOPs of exactly the sampled rows."""
    from paper_2506_02965_amd.synth import make_inputs
    cfg = LayerConfig("cb", T=64, d=128, f=128, E=4, k=2, seed=3)
    inp = make_inputs(cfg, with_dy=True)
    out = bench.cpu_baseline(cfg, inp, min_seconds=0.0, max_seconds=60.0)
    assert out["kind"] == "oracle" and out["unit"] == "TFLOP/s" and out["value"] > 0
    assert "1 of the 4 experts" in out["sample"]
    rows = int(out["sample"].split("(")[1].split(" ")[0])
    assert abs(out["sample_gflop"] * 1e9 - (2 * 64 * 128 * 4 + 18 * 128 * 128 * rows)) < 1e8
