"""Benchmark of the MoE expert layer (forward + backward) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step is one pass of the whole layer over one batch of resident synthetic inputs:
route -> permute -> expert FFN forward -> combine -> combine backward -> expert FFN backward
-> router backward -> unpermute. The workload is the bf16 layer T=4096, d=1024, f=2816,
E=16 SwiGLU experts, top-2 (seeded inputs, weights ~ N(0, 1/fan_in)).

Prints ONE JSON line: the layer's algorithmic TFLOP/s (6*d*f per routed-or-shared row forward,
12*d*f backward, 2*T*d*E router forward, 4*T*d*E router backward), tokens/s, the roofline of the
dominant kernel (found in the last two warm-up steps) measured with HIP events recorded by the library
around that kernel only, on its launch stream, during the timed steps, and the CPU oracle's throughput on
the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2516.6      # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 FLOP/clk
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 matrix
HBM_PEAK_GBS = 8000.0

# algorithmic FLOPs of each kernel per launch, per routed-or-shared row (x d*f)
GEMM_FLOPS_PER_ROW_DF = {
    "gemm_fwd_gate_up": 4.0, "gemm_fwd_down": 2.0, "gemm_bwd_dh": 2.0, "gemm_wgrad_down": 2.0,
    "gemm_wgrad_gate_up": 4.0, "gemm_bwd_dx": 4.0,
    # two independent contractions in one launch
    "gemm_bwd_dh+wgrad_down": 4.0, "gemm_bwd_dx+wgrad_gate_up": 8.0,
}


COPY_CAL_BYTES = 256 << 20   # bytes read (and written) by one calibration copy
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_dominant_kernel.txt")
GEMM_SOURCES = [os.path.join(ROOT, "paper_2506_02965_amd", "csrc", n)
                for n in ("grouped_gemm_bf16.hip", "grouped_gemm.h", "pcmoe_internal.h")]


def gemm_source_digest():
    h = hashlib.sha256()
    for path in GEMM_SOURCES:
        with open(path, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the FETCH_SIZE / WRITE_SIZE counter passes recorded in
    TRAFFIC_FILE, each scaled by what the same counter reads for the calibration copy of known size;
    None when no record matches this kernel, workload and the current GEMM sources."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    rec = {}
    with open(TRAFFIC_FILE) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    try:
        if rec["kernel"] != kernel or rec["workload"] != workload or rec["gemm_sources"] != gemm_source_digest():
            return None
        cal_kib = COPY_CAL_BYTES / 1024.0
        fetch = float(rec["fetch_kib_per_launch"]) * cal_kib / float(rec["copy_fetch_kib"])
        write = float(rec["write_kib_per_launch"]) * cal_kib / float(rec["copy_write_kib"])
    except (KeyError, ValueError, ZeroDivisionError):
        return None
    return round((fetch + write) * 1024.0)


def layer_flops(cfg, n_routed_rows, backward=True):
    rows = n_routed_rows + cfg.n_shared * cfg.T
    fl = 6.0 * cfg.d * cfg.f * rows + 2.0 * cfg.T * cfg.d * cfg.E
    if backward:
        fl += 12.0 * cfg.d * cfg.f * rows
        if cfg.router_backward:
            fl += 4.0 * cfg.T * cfg.d * cfg.E
    return fl


def cpu_baseline(cfg, inp, min_seconds=10.0, max_seconds=30.0):
    """The CPU oracle (fp64 numpy) on this host's cores, timed on a bounded sample of the workload:
    whole forward + backward passes of the layer, repeated until about min_seconds of CPU work
    (first pass always counted; no new pass starts beyond max_seconds)."""
    from oracle import moe_layer as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    n_pass, total, n_rows = 0, 0.0, 0
    while True:
        t0 = time.perf_counter()
        fwd = O.layer_forward(inp)
        O.layer_backward(inp, fwd, inp.dy)
        total += time.perf_counter() - t0
        n_pass += 1
        n_rows = len(fwd["row_to_slot"])
        if total >= min_seconds or total * (n_pass + 1) / n_pass > max_seconds:
            break
    dt = total / n_pass
    fl = layer_flops(cfg, n_rows, True)
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n_pass} whole fwd+bwd pass(es) of the workload ({cfg.T} tokens), fp64 numpy, "
                      f"{total:.1f} s in total", "tokens_per_s": round(cfg.T / dt, 2), "seconds_per_pass": round(dt, 3)}


def measure_expert_update(P, layer, w, steps):
    """The expert update (AdamW with an fp32 master copy) over the hosted experts, timed on its own
    after the layer steps: HBM bytes per launch = parameters x (weight written 2, gradient read 2, master
    4+4, moments 8+8) for bf16 weights. With a master copy the stored weight is only written: the update
    reads the fp32 master instead."""
    import torch
    layer.init_update_state(w, master=True)
    opt = P.make_opt(kind="adamw", lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    for _ in range(2):
        layer.update(w, opt)
    torch.cuda.synchronize()
    P.moe_kernel_timing_select("expert_update")
    P.moe_kernel_timing(True)
    n = max(steps // 2, 3)
    for _ in range(n):
        layer.update(w, opt)
    torch.cuda.synchronize()
    cnt, ms = P.moe_kernel_timing_report()["expert_update"]
    P.moe_kernel_timing(False)
    P.moe_kernel_timing_select(None)
    params = layer.opt_m.numel()
    es = w.w_gate.element_size()
    per_param = 2 * es + 8 + 16           # weight written, gradient read; master and moments read+write
    avg_s = ms / cnt / 1e3
    gbs = params * per_param / avg_s / 1e9
    return {"kernel": "expert_update", "optimizer": "adamw, fp32 master", "parameters": params,
            "bytes_per_launch": params * per_param, "avg_launch_us": round(avg_s * 1e6, 2),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(gbs / HBM_PEAK_GBS, 4)}}


def hbm_steps(cfg, n_routed, kernels):
    """Achieved HBM bandwidth of the bandwidth-bound steps from their algorithmic bytes per launch
    (s = element bytes, N = routed rows, S = shared experts):
      router forward   T*d*s + E*d*s + 4*T*E + 8*T*k   (x and W_r read; logits, top-k indices and weights written)
      permute          T*d*s + N*d*s + 8*T*k           (histogram, scatter and gather launches together)
      combine          N*d*s + T*d*s + S*T*d*s + 8*T*k
      combine backward T*d*s + 2*N*d*s + 8*T*k
      unpermute        N*d*s + T*d*s + S*T*d*s + 4*T*k
    The times are the warm-up steps' HIP events around every launch, which include the gap between
    back-to-back launches (about 1-2 us here), so the rates are lower bounds of the kernels' own."""
    s = 2 if cfg.dtype == "bf16" else 4
    T, d, k, E, S, N = cfg.T, cfg.d, cfg.k, cfg.E, cfg.n_shared, n_routed
    table = {
        "route_fwd": (("route_fwd",), T * d * s + E * d * s + 4 * T * E + 8 * T * k),
        "permute": (("permute_hist", "permute_scatter", "permute_gather"), T * d * s + N * d * s + 8 * T * k),
        "combine": (("combine",), N * d * s + T * d * s + S * T * d * s + 8 * T * k),
        "combine_bwd": (("combine_bwd",), T * d * s + 2 * N * d * s + 8 * T * k),
        "unpermute": (("unpermute",), N * d * s + T * d * s + S * T * d * s + 4 * T * k),
    }
    out = {}
    for step, (names, nbytes) in table.items():
        if not all(n in kernels for n in names):
            continue
        us = sum(kernels[n]["avg_us"] for n in names)
        gbs = nbytes / (us * 1e-6) / 1e9
        out[step] = {"bytes": nbytes, "us": round(us, 2), "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}
    return out


def memory_amortisation(P, parties=(1, 2, 4, 8)):
    """The per-party memory claim of Sec. 3 (experts sharded over n parties): one party's peak device memory for
    the expert layer's training step when it hosts all E experts or E/n of them. The row-space buffers keep their
    capacity of T*k rows either way, which is what a host receives in expectation from all parties under uniform
    routing. A shard cannot run the router adjoint (it needs every host's gate gradients), so that one kernel is
    skipped for n > 1 while its buffers stay allocated. Synthetic inputs; no model or dataset."""
    import dataclasses
    import torch
    from paper_2506_02965_amd.layer import MoELayer, upload, training_footprint
    from paper_2506_02965_amd.synth import make_inputs
    base = dataclasses.replace(CONFIGS[3], bias=None, router_backward=True, local_begin=0)
    rows = []
    for n in parties:
        cfg = dataclasses.replace(base, local_count=base.E // n)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        start = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        inp = make_inputs(cfg, with_dy=True)
        w = upload(inp)
        del inp
        layer = MoELayer(cfg, backward=True, router_backward=True)
        layer.init_update_state(w, master=True)
        layer.dlogits.zero_()
        layer.forward(w)
        layer.combine_bwd(w.dy)
        layer.ffn_bwd(w, w.dy)
        if n == 1:
            layer.route_bwd(w)
        layer.permute_bwd(w)
        layer.update(w, P.make_opt(kind="adamw", lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1))
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated() - start
        acc = training_footprint(cfg, cfg.n_local)
        rows.append({"parties": n, "hosted_experts": cfg.n_local, "measured_peak_bytes": int(peak),
                     "accounted_bytes": acc["total"], "expert_state_bytes": acc["expert_state"],
                     "activation_bytes": acc["activations"], "owner_bytes": acc["owner"]})
        del layer, w
    full = rows[0]["measured_peak_bytes"]
    for r in rows:
        r["relative_to_all_experts"] = round(r["measured_peak_bytes"] / full, 4)
    return {"experiment": "per-party memory of the expert layer's training step, experts sharded over n parties",
            "workload": "T=8192 d=2048 f=1408 E=64 top-4, bf16, AdamW with fp32 master and moments",
            "data": "synthetic", "rows": rows}


def pick_workload(key: str):
    from paper_2506_02965_amd.synth import CONFIGS
    for i, c in CONFIGS.items():
        if key in (c.name, str(i)):
            return c
    raise SystemExit(f"unknown workload {key!r}; known: " + ", ".join(c.name for c in CONFIGS.values()))


def main():
    from paper_2506_02965_amd.synth import CONFIGS
    WORKLOADS = list(CONFIGS.values())
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # The first ~60 steps (~50 ms) of a fresh process run up to 7% slower than the steady state that follows;
    # the default warm-up covers them.
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", "--config", dest="workload", default="bf16_T4096_d1024_f2816_E16_k2",
                    help="workload name (" + ", ".join(c.name for c in WORKLOADS) + ") or its position 1-5 in that list")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--memory", action="store_true",
                    help="instead of the benchmark: peak device memory of one party's expert-layer training step "
                         "(fwd, bwd, AdamW update) hosting all 64 experts of the T=8192/d=2048/f=1408/E=64/k=4 "
                         "layer or 1/n of them (n = 2, 4, 8 parties), measured and accounted")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="before the warm-up, copy a 256 MiB device buffer three times (the reference kernel "
                         "that scales the HBM byte counters of a rocprofv3 --pmc run)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the layer is one party's shard on one MI355X; "
              "multi-GPU expert sharding is not built", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2506_02965_amd import pcmoe as P
    from paper_2506_02965_amd.layer import MoELayer, upload
    from paper_2506_02965_amd.synth import make_inputs

    P.lib()
    if args.memory:
        print(json.dumps(memory_amortisation(P)), flush=True)
        return
    if args.copy_calibration:
        src = torch.ones(COPY_CAL_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cfg = pick_workload(args.workload)
    inp = make_inputs(cfg, with_dy=True)
    w = upload(inp, device="cuda")
    layer = MoELayer(cfg, backward=True)

    def step():
        layer.forward(w)
        layer.backward(w)

    for _ in range(max(args.warmup - 2, 0)):
        step()
    torch.cuda.synchronize()
    n_routed = layer.n_local_rows()
    # the last two warm-up steps record every kernel to find the dominant one (untimed)
    P.moe_kernel_timing(True)
    for _ in range(min(args.warmup, 2)):
        step()
    torch.cuda.synchronize()
    kt_all = P.moe_kernel_timing_report()
    P.moe_kernel_timing(False)
    dom_name = max(kt_all.items(), key=lambda kv: kv[1][1])[0]

    # timed steps: HIP events only around the dominant kernel, on the stream it is launched on
    P.moe_kernel_timing_select(dom_name)
    P.moe_kernel_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / args.steps
    kt = P.moe_kernel_timing_report()
    P.moe_kernel_timing(False)
    P.moe_kernel_timing_select(None)

    flops = layer_flops(cfg, n_routed, True)
    tflops = flops / dt / 1e12
    rows = n_routed + cfg.n_shared * cfg.T
    dom_cnt, dom_ms = kt[dom_name]
    dom_avg_s = dom_ms / dom_cnt / 1e3
    nw = min(args.warmup, 2)
    kernels = {k: {"launches_per_step": c / nw, "avg_us": ms / c * 1e3} for k, (c, ms) in kt_all.items()}
    if dom_name in GEMM_FLOPS_PER_ROW_DF:
        per_launch = GEMM_FLOPS_PER_ROW_DF[dom_name] * cfg.d * cfg.f * rows
        ach = per_launch / dom_avg_s / 1e12
        peak = BF16_PEAK_TFLOPS if cfg.dtype == "bf16" else FP32_PEAK_TFLOPS
        roof = {"kernel": dom_name, "bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4), "traffic": measured_traffic(dom_name, cfg.name),
                "algorithmic_per_launch": per_launch, "avg_launch_us": round(dom_avg_s * 1e6, 2)}
    else:
        roof = {"kernel": dom_name, "bound": None, "achieved": None, "peak": None, "unit": None, "frac": None,
                "traffic": None, "avg_launch_us": round(dom_avg_s * 1e6, 2)}
    gemm_us = sum(v["avg_us"] * v["launches_per_step"] for k, v in kernels.items() if k.startswith("gemm_"))
    out = {
        "metric": "MoE-layer fwd+bwd TFLOP/s and tokens/s; % of MI355X bf16 MFMA peak",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,1) activations, N(0,1/fan_in) weights)",
        "config": {"workload": cfg.name, "T": cfg.T, "d_model": cfg.d, "d_ff": cfg.f, "E": cfg.E, "top_k": cfg.k,
                   "n_shared": cfg.n_shared, "hosted_experts": cfg.n_local, "routed_rows": n_routed,
                   "parallelism": "single GPU"},
        "tokens_per_s": round(cfg.T / dt, 1),
        "pct_bf16_peak": round(100.0 * tflops / BF16_PEAK_TFLOPS, 3),
        "expert_gemm_tflops": round((18.0 * cfg.d * cfg.f * rows) / (gemm_us * 1e-6) / 1e12, 2) if gemm_us else None,
        "roofline": roof,
        "kernels_warmup": {k: {"avg_us": round(v["avg_us"], 2), "per_step": v["launches_per_step"]}
                           for k, v in kernels.items()},
        "hbm_steps_warmup": hbm_steps(cfg, n_routed, kernels),
    }
    out["expert_update"] = measure_expert_update(P, layer, w, args.steps)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, inp)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
