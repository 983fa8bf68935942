"""Benchmark of the MoE expert layer (forward + backward) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step is one pass of the whole layer over one batch of resident synthetic inputs:
route -> permute -> expert FFN forward -> combine -> combine backward -> expert FFN backward
-> router backward -> unpermute. The default workload is the largest one, the bf16 layer T=8192,
d=4096, f=14336, E=8 SwiGLU experts, top-2 (seeded inputs, weights ~ N(0, 1/fan_in)); --workload
selects another.

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


def host_info():
    """What the CPU baseline ran on: the cores this process may use, the CPU model, the BLAS library numpy calls
    and its thread count (the threads the oracle's matrix products actually use)."""
    import numpy as np
    np.ones((64, 64)) @ np.ones((64, 64))             # loads the BLAS so that its thread pool is reported
    blas, threads = "unknown", None
    try:
        from threadpoolctl import threadpool_info
        pools = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if pools:
            blas = f"{pools[0].get('internal_api')} {pools[0].get('version')} ({pools[0].get('threading_layer')})"
            threads = max(int(i.get("num_threads", 1)) for i in pools)
    except Exception:
        pass
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    avail = len(os.sched_getaffinity(0))
    return {"cores_available": avail, "cpu_model": model, "blas": blas, "blas_threads": threads or avail}


def cpu_baseline(cfg, inp, min_seconds=10.0, max_seconds=30.0):
    """The CPU oracle (fp64 numpy) on this host's cores, timed on a bounded sample of the workload: the oracle's
    routing and dispatch of every token (scores, top-k, gate weights, the permutation), then its forward and
    backward of one expert at a time over that expert's rows (hosted experts in order, then shared ones), the
    per-expert steps of the whole-layer oracle, until about min_seconds of CPU work (at least one expert; no
    expert starts that would end past max_seconds by the last one's time). Throughput = the algorithmic FLOPs
    of the sampled work (router forward 2*T*d*E, 18*d*f per expert row) / its time."""
    import numpy as np
    from oracle import moe_layer as O
    info = host_info()
    T, d, f, E, k = cfg.T, cfg.d, cfg.f, cfg.E, cfg.k
    t0 = time.perf_counter()
    L64 = O.router_logits(inp.x, inp.w_router, inp.logit_bias, cfg.bias_groups)
    idx = O.topk_indices(O.selection_logits(L64), k)
    w = O.gate_weights(L64, idx, renormalize=cfg.renormalize)
    counts, offsets, r2s, s2r = O.permutation(idx, cfg.local_begin, cfg.n_local)
    flops = 2.0 * T * d * E
    elapsed = time.perf_counter() - t0
    x64, dy64, wflat = np.asarray(inp.x, np.float64), np.asarray(inp.dy, np.float64), w.reshape(-1)
    done, rows_done, last = 0, 0, 0.0
    for g in range(cfg.n_groups):
        if done and (elapsed >= min_seconds or elapsed + last > max_seconds):
            break
        t1 = time.perf_counter()
        if g < cfg.n_local:
            rr = r2s[offsets[g]:offsets[g + 1]]
            tok = rr // k
            h, dO = x64[tok], wflat[rr][:, None] * dy64[tok]
        else:
            h, dO = x64, dy64
        if len(h):
            G, U, Hd, _ = O.expert_forward(h, inp.w_gate[g], inp.w_up[g], inp.w_down[g])
            O.expert_backward(h, inp.w_gate[g], inp.w_up[g], inp.w_down[g], G, U, Hd, dO)
        last = time.perf_counter() - t1
        elapsed += last
        flops += 18.0 * d * f * len(h)
        rows_done += len(h)
        done += 1
    out = {"value": flops / elapsed / 1e12, "unit": "TFLOP/s", "cores": int(info["blas_threads"]), "kind": "oracle",
           "sample": f"routing and dispatch of all {T} tokens, then forward + backward of {done} of the "
                     f"{cfg.n_groups} experts ({rows_done} expert rows), fp64 numpy, {elapsed:.1f} s",
           "sample_seconds": round(elapsed, 2), "sample_gflop": round(flops / 1e9, 1)}
    out.update(info)
    return out


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


def dense_reference(cfg, steps=20):
    """Context, not a target: the vendor's dense bf16 GEMM (torch.matmul, i.e. hipBLASLt) on the workload's expert
    contractions with all routed rows as one dense matrix (forward gate|up, forward down, input gradient dX).
    TFLOP/s per shape, timed with HIP events on random bf16 operands."""
    import torch
    rows = cfg.T * cfg.k
    shapes = [("gate_up", rows, cfg.d, 2 * cfg.f), ("down", rows, cfg.f, cfg.d), ("dx", rows, 2 * cfg.f, cfg.d)]
    out = {}
    for name, M, K, N in shapes:
        a = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
        b = torch.randn(N, K, device="cuda", dtype=torch.bfloat16)
        for _ in range(3):
            a @ b.t()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            a @ b.t()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / steps
        tf = 2.0 * M * K * N / us / 1e6
        out[name] = {"M": M, "K": K, "N": N, "us": round(us, 1), "TFLOP/s": round(tf, 1),
                     "frac": round(tf / BF16_PEAK_TFLOPS, 4)}
        del a, b
    return {"dense_reference": "torch.matmul (hipBLASLt), bf16", "workload": cfg.name, "shapes": out}


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


DEFAULT_WORKLOAD = "bf16_T8192_d4096_f14336_E8_k2"


def progress(msg):
    """A progress line on stderr (stdout carries only the JSON line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


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
    # the warm-up runs at least --warmup steps and at least --min-warmup-seconds.
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--min-warmup-seconds", type=float, default=2.0)
    ap.add_argument("--workload", "--config", dest="workload", default=DEFAULT_WORKLOAD,
                    help="workload name (" + ", ".join(c.name for c in WORKLOADS) + ") or its position 1-5 in that list")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--memory", action="store_true",
                    help="instead of the benchmark: peak device memory of one party's expert-layer training step "
                         "(fwd, bwd, AdamW update) hosting all 64 experts of the T=8192/d=2048/f=1408/E=64/k=4 "
                         "layer or 1/n of them (n = 2, 4, 8 parties), measured and accounted")
    ap.add_argument("--dense-reference", action="store_true",
                    help="instead of the benchmark: the vendor's dense bf16 GEMM (torch.matmul) on the workload's "
                         "gate|up, down and dX shapes with all routed rows as one matrix (context for the roofline)")
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
    if args.dense_reference:
        print(json.dumps(dense_reference(pick_workload(args.workload))), flush=True)
        return
    if args.copy_calibration:
        src = torch.ones(COPY_CAL_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cfg = pick_workload(args.workload)
    progress(f"workload {cfg.name}: drawing the inputs")
    inp = make_inputs(cfg, with_dy=True)
    w = upload(inp, device="cuda")
    layer = MoELayer(cfg, backward=True)
    progress("inputs resident on the GPU; warm-up")

    def step():
        layer.forward(w)
        layer.backward(w)

    warm_steps, t_warm = 0, time.perf_counter()
    while warm_steps < max(args.warmup - 2, 0) or time.perf_counter() - t_warm < args.min_warmup_seconds:
        step()
        warm_steps += 1
        if warm_steps % 8 == 0:
            torch.cuda.synchronize()   # the host stays at most a few steps ahead, so the clock measures the GPU
    torch.cuda.synchronize()
    warm_steps += 2
    n_routed = layer.n_local_rows()
    # the last two warm-up steps record every kernel to find the dominant one (untimed)
    P.moe_kernel_timing(True)
    for _ in range(2):
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
    nw = 2
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
        "warmup_steps_run": warm_steps,
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
        progress("GPU steps done; timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(cfg, inp)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
