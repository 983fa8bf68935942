"""Parity of the HIP layer (through the C ABI) with the CPU oracle on the GPU.

Small cases run the whole oracle and compare every output element by element; they span several
GEMM tiles and ragged tails. The five workloads run at full size in the launch configuration the
benchmark times; the two largest (T=8192 d=4096 f=14336, and T=16384 with 64 experts) are checked in full
against the oracle evaluated one expert group at a time. Routing indices and the permutation are bit-exact
everywhere."""
import dataclasses
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

from paper_2506_02965_amd.synth import CONFIGS, LayerConfig, make_inputs
from gpu_util import check_full, check_full_streamed, run_gpu, log

pytestmark = pytest.mark.gpu


def small_cases():
    C = {}
    C["fp32_T512_full"] = (CONFIGS[1], None)
    C["f32_fwd_bwd_shared"] = (LayerConfig("f32b", T=300, d=256, f=384, E=8, k=2, n_shared=1, dtype="f32",
                                           seed=10), None)
    C["bf16_T1000_E16"] = (LayerConfig("c2s", T=1000, d=256, f=384, E=16, k=2, seed=11), None)
    C["shard_E64_loc16"] = (LayerConfig("c3s", T=1024, d=256, f=256, E=64, k=4, local_begin=0, local_count=16,
                                        router_backward=False, bias="party", parties=4, seed=12), None)
    C["shard_E64_loc16_mid"] = (LayerConfig("c3m", T=1024, d=256, f=256, E=64, k=4, local_begin=16,
                                            local_count=16, router_backward=False, bias="party", parties=4,
                                            seed=12), None)
    C["bf16_d512_f1024_E8"] = (LayerConfig("c4s", T=512, d=512, f=1024, E=8, k=2, seed=13), None)
    C["E64_k6_shared_zipf"] = (LayerConfig("c5s", T=1024, d=256, f=384, E=64, k=6, n_shared=2, bias="zipf",
                                              seed=14), None)
    C["renormalize0"] = (LayerConfig("r0", T=512, d=256, f=256, E=16, k=4, renormalize=False, seed=15), None)
    C["k1"] = (LayerConfig("k1", T=256, d=128, f=128, E=4, k=1, seed=16), None)
    C["k_equals_E"] = (LayerConfig("kE", T=256, d=128, f=128, E=4, k=4, seed=17), None)
    C["T1"] = (LayerConfig("t1", T=1, d=128, f=128, E=8, k=2, n_shared=1, seed=18), None)
    # many experts (router tiles of 8 and 16 expert blocks), k at its maximum, d not a multiple of 512
    C["E200_k8_d384"] = (LayerConfig("e200", T=512, d=384, f=256, E=200, k=8, seed=23), None)
    C["E128_f32"] = (LayerConfig("e128", T=256, d=256, f=128, E=128, k=2, dtype="f32", seed=24), None)
    C["E24_k3"] = (LayerConfig("e24", T=300, d=512, f=256, E=24, k=3, n_shared=1, seed=25), None)
    # the largest supported shapes of the routing and of the tile plan: E = 256 experts, k = 8, and 511 groups
    # (256 hosted + 255 shared experts), most of them with a handful of rows
    C["E256_k8_511_groups"] = (LayerConfig("g511", T=64, d=128, f=128, E=256, k=8, n_shared=255, seed=31), None)

    def forced_empty(inp):
        inp.logit_bias[0, 3] = -1e4
        inp.logit_bias[0, 7] = -1e4
    C["forced_empty_experts"] = (LayerConfig("fe", T=512, d=256, f=256, E=8, k=2, bias="forced_empty", seed=19),
                                 forced_empty)

    # a party whose hosted experts (4..7) receive no token: every routed group of its grouped GEMMs is empty
    # (N_loc = 0), alone and beside a shared expert
    def no_hosted_tokens(inp):
        inp.logit_bias[0, 4:8] = -1e4
    C["shard_without_tokens"] = (LayerConfig("nt", T=512, d=256, f=256, E=8, k=2, local_begin=4, local_count=4,
                                             router_backward=False, bias="forced_empty", seed=27), no_hosted_tokens)
    C["shard_without_tokens_shared"] = (LayerConfig("nts", T=512, d=256, f=256, E=8, k=2, local_begin=4,
                                                    local_count=4, n_shared=1, router_backward=False,
                                                    bias="forced_empty", seed=28), no_hosted_tokens)

    def all_to_one(inp):
        inp.logit_bias[0, 2] = 1e4
    C["all_tokens_one_expert"] = (LayerConfig("a1", T=384, d=128, f=256, E=4, k=1, bias="forced_empty", seed=20),
                                  all_to_one)

    # Expert row counts set through a per-token logit bias: remainders 0, 1, 64, 65, 128, 129 and 255 of the
    # 256-row m-tiles, an empty expert, and more 256 x 256 tiles than CUs in the gate/up contraction
    # (tail m-tiles of at most 128 rows scheduled after the others).
    tail_counts = [0, 1, 320, 321, 384, 385, 511, 1174, 1000]

    def forced_counts(inp):
        T = inp.cfg.T
        slots = np.repeat(np.arange(len(tail_counts)), tail_counts)  # 2T slots, sorted by expert
        assert slots.size == 2 * T
        inp.logit_bias[:] = -1e4
        t = np.arange(T)
        inp.logit_bias[t, slots[:T]] = 2e4  # first choice
        inp.logit_bias[t, slots[T:]] = 1e4  # second choice: another expert (no count exceeds T)
    C["tail_tiles_forced_counts"] = (LayerConfig("tt", T=2048, d=256, f=2048, E=len(tail_counts), k=2, bias="party",
                                                 parties=2048, seed=26), forced_counts)

    # d_model = 4096 selects the software-pipelined one-wavefront-per-SIMD tile for every contraction but the down
    # projection: ragged tail m-tiles (about 150 rows per expert, 600 shared-expert rows), a last n-tile of 128
    # columns (f = 384), weight gradients with an odd number of 32-deep K-tiles, and groups with no rows at all
    C["pipelined_d4096_ragged_shared"] = (LayerConfig("p4", T=600, d=4096, f=384, E=8, k=2, n_shared=1, seed=32), None)

    def two_empty(inp):
        inp.logit_bias[0, 1] = -1e4
        inp.logit_bias[0, 6] = -1e4
        inp.logit_bias[0, 3] = 3.0  # one heavy expert: several m-tiles
    C["pipelined_d4096_empty_experts"] = (LayerConfig("p4e", T=512, d=4096, f=256, E=8, k=2, bias="forced_empty",
                                                      seed=33), two_empty)

    # d_model = 4096 with enough weight-gradient tiles (9 groups x 32 x 16 and 9 x 16 x 16) that both backward
    # launches run their weight gradients in persistent workgroups by default, beside a shared expert
    C["pipelined_persistent_default"] = (LayerConfig("pp", T=1024, d=4096, f=4096, E=8, k=2, n_shared=1, seed=34),
                                         None)
    # a down projection of 384 tiles of 256 x 256 (one and a half rounds of the chip) and three tail m-tiles of 22,
    # 33 and 50 rows: each of the 24 tail tiles runs as four 64-column windows
    C["down_tail_split"] = (LayerConfig("dts", T=4096, d=2048, f=512, E=8, k=2, n_shared=1, seed=35), None)
    # 13 tail m-tiles (1 to 37 rows) over 8 n-tiles: four windows each would not fit the chip's 256 CUs, so the
    # decode takes two per tail tile
    C["down_tail_split_fewer_windows"] = (LayerConfig("dtw", T=4096, d=2048, f=512, E=32, k=4, seed=37), None)

    def zero_router(inp):
        inp.w_router[:] = 0
    C["ties_all_equal"] = (LayerConfig("z", T=256, d=128, f=128, E=8, k=3, seed=21), zero_router)

    def dup_router(inp):
        inp.w_router[5] = inp.w_router[2]
        inp.w_router[6] = inp.w_router[2]
    C["ties_duplicate_rows"] = (LayerConfig("dup", T=256, d=128, f=128, E=8, k=3, seed=22), dup_router)
    return C


SMALL = small_cases()


@pytest.mark.parametrize("name", list(SMALL))
def test_layer_small(name):
    cfg, edit = SMALL[name]
    log(f"[parity] {name}: T={cfg.T} d={cfg.d} f={cfg.f} E={cfg.E} k={cfg.k} S={cfg.n_shared} {cfg.dtype}")
    inp = make_inputs(cfg, with_dy=True)
    if edit:
        edit(inp)
    layer, _ = run_gpu(cfg, inp)
    errs = check_full(cfg, inp, layer)
    log(f"[parity] {name}: " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))


def run_small_bf16_cases(tag):
    """Every bf16 small case, in this process (the child of the tests below); the first case runs twice and its
    outputs must be bit-identical (tiles claimed at run time change which CU computes a tile, not its result)."""
    for n, (name, (cfg, edit)) in enumerate((k, v) for k, v in SMALL.items() if v[0].dtype == "bf16"):
        inp = make_inputs(cfg, with_dy=True)
        if edit:
            edit(inp)
        layer, _ = run_gpu(cfg, inp)
        errs = check_full(cfg, inp, layer)
        if n == 0:
            again, _ = run_gpu(cfg, inp)
            for t in ("y", "dgate", "dw_gate", "dw_up", "dw_down", "dx"):
                assert torch.equal(getattr(layer, t), getattr(again, t)), f"{name}: {t} differs between runs"
        log(f"[parity, {tag}] {name}: max rel err {max(errs.values()):.2e}")


def run_small_in_child(tag, **env_over):
    """The bf16 small cases in one child process with environment overrides (read once per process)."""
    here = os.path.dirname(os.path.abspath(__file__))
    env = dict(os.environ, **env_over)
    code = (f"import sys; sys.path.insert(0, {os.path.dirname(here)!r}); sys.path.insert(0, {here!r}); "
            f"import test_gpu_parity as T; T.run_small_bf16_cases({tag!r})")
    log(f"[parity] small bf16 cases, {tag} (child process)")
    r = subprocess.run([sys.executable, "-u", "-c", code], env=env, capture_output=True, text=True, timeout=380)
    log(r.stdout[-4000:])
    assert r.returncode == 0, r.stderr[-4000:]
    assert r.stdout.count(f"[parity, {tag}]") == sum(c.dtype == "bf16" for c, _ in SMALL.values())


@pytest.mark.timeout(400)
def test_layer_small_pipelined_tile_forced():
    """The bf16 small cases again with the software-pipelined one-wavefront-per-SIMD tile forced on all six
    contractions (by default it is chosen only at d_model >= 4096): ragged and empty groups, tails, E = 256 with 511
    groups, ragged last n-tiles; the paired launches run their weight gradients in persistent workgroups and the
    gate/up launch claims its last tiles by ticket (by default only when those fill 8 rounds of the chip)."""
    run_small_in_child("pipelined tile forced", PCMOE_GEMM_TILES=",".join(f"{k}=256x256w4" for k in range(6)),
                       PCMOE_DYN="2")


@pytest.mark.timeout(400)
def test_layer_small_pipelined_tile_ticket_tails():
    """As above, with the pipelined paired launches' weight gradients on ticket-claimed tails instead of persistent
    workgroups (PCMOE_PERSIST=0)."""
    run_small_in_child("pipelined tile, ticket tails", PCMOE_GEMM_TILES=",".join(f"{k}=256x256w4" for k in range(6)),
                       PCMOE_DYN="2", PCMOE_PERSIST="0")


@pytest.mark.timeout(400)
def test_layer_small_ticket_tiles_forced():
    """The bf16 small cases with the default tiles and ticket-claimed weight-gradient tiles in every paired launch,
    down to groups with a single tile."""
    run_small_in_child("ticket tiles forced", PCMOE_DYN="2")


def test_deterministic_bits():
    """Two runs of the same layer give bit-identical outputs (fixed reduction orders, no atomics)."""
    cfg = LayerConfig("det", T=1000, d=256, f=384, E=16, k=2, n_shared=1, seed=23)
    inp = make_inputs(cfg, with_dy=True)
    a, _ = run_gpu(cfg, inp)
    b, _ = run_gpu(cfg, inp)
    for n in ("logits", "topk_idx", "row_to_slot", "slot_to_row", "y", "dgate", "dw_gate", "dw_up", "dw_down",
              "dw_router", "dx"):
        assert torch.equal(getattr(a, n), getattr(b, n)), n


@pytest.mark.parametrize("c", [1, 2, 3], ids=lambda c: CONFIGS[c].name)
def test_workload_full_size(c):
    cfg = CONFIGS[c]
    log(f"[parity] full-size workload {cfg.name}")
    inp = make_inputs(cfg, with_dy=True)
    layer, _ = run_gpu(cfg, inp)
    errs = check_full(cfg, inp, layer)
    log(f"[parity] {cfg.name}: " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("c", [4, 5], ids=lambda c: CONFIGS[c].name)
def test_workload_full_size_streamed(c):
    cfg = CONFIGS[c]
    log(f"[parity] full-size workload {cfg.name} (oracle one expert group at a time)")
    inp = make_inputs(cfg, with_dy=True)
    log(f"[parity] {cfg.name}: inputs drawn")
    layer, _ = run_gpu(cfg, inp)
    log(f"[parity] {cfg.name}: GPU layer done")
    errs = check_full_streamed(cfg, inp, layer)
    log(f"[parity] {cfg.name}: " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
