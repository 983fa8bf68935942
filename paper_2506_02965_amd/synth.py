"""Seeded synthetic inputs for the MoE expert layer.

This module is shared by the HIP path's tests/bench and by the CPU oracle's tests. It holds
no step of the layer's arithmetic: it only draws tensors, rounds them to the storage
precision and describes the five workload shapes.

Workloads (shapes stand in for the paper's fine-tuning runs, whose model, data and layer sizes
are not published; Sec. 4 setup, Table 1):

  1  fp32 forward only,  T=512,  d=256,  f=512,   E=8,  top-2
  2  bf16 fwd+bwd,       T=4096, d=1024, f=2816,  E=16, top-2 (the benchmark's workload)
  3  bf16 fwd+bwd shard, T=8192 (4 parties x 2048), d=2048, f=1408, E=64 global,
     this GPU hosts experts 0..15, top-4, per-party N(0,1) logit bias
  4  bf16 fwd+bwd,       T=8192, d=4096, f=14336, E=8,  top-2
  5  bf16 fwd+bwd,       T=16384, d=2048, f=1408, E=64 routed top-6 + 2 shared experts,
     logit bias log p_e with p ~ Zipf(s=1.1) over experts

Draw recipe: every tensor has its own numpy PCG64 stream keyed by (seed, tag, expert), drawn
as float32 standard normals, scaled in float32, and for bf16 workloads rounded once to
bf16 (round-to-nearest-even). x ~ N(0,1); dY ~ N(0,1); router and gate/up weights
~ N(0, 1/d); down weights ~ N(0, 1/f) (variance 1/fan_in).
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

# stream tags, one per tensor kind
TAG_X, TAG_DY, TAG_WG, TAG_GATE, TAG_UP, TAG_DOWN, TAG_BIAS, TAG_SH_GATE, TAG_SH_UP, TAG_SH_DOWN = range(10)


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    T: int
    d: int
    f: int
    E: int
    k: int
    local_begin: int = 0
    local_count: Optional[int] = None   # None = all E experts hosted here
    n_shared: int = 0
    dtype: str = "bf16"                 # storage dtype: "f32" or "bf16"
    backward: bool = True
    router_backward: bool = True        # False for a party shard: the data owner differentiates the router
    bias: Optional[str] = None          # None | "party" | "zipf" | "forced_empty"
    parties: int = 1
    renormalize: bool = True
    seed: int = 0

    @property
    def n_local(self) -> int:
        return self.E if self.local_count is None else self.local_count

    @property
    def n_groups(self) -> int:
        return self.n_local + self.n_shared

    @property
    def bias_groups(self) -> int:
        if self.bias == "party":
            return self.parties
        return 1

    def scaled(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    1: LayerConfig("fp32_fwd_T512_d256_f512_E8_k2", T=512, d=256, f=512, E=8, k=2,
                   dtype="f32", backward=False, seed=0),
    2: LayerConfig("bf16_T4096_d1024_f2816_E16_k2", T=4096, d=1024, f=2816, E=16, k=2, seed=1),
    3: LayerConfig("bf16_shard_T8192_d2048_f1408_E64loc16_k4", T=8192, d=2048, f=1408, E=64, k=4,
                   local_begin=0, local_count=16, router_backward=False, bias="party", parties=4, seed=2),
    4: LayerConfig("bf16_T8192_d4096_f14336_E8_k2", T=8192, d=4096, f=14336, E=8, k=2, seed=3),
    5: LayerConfig("bf16_T16384_d2048_f1408_E64_k6_S2", T=16384, d=2048, f=1408, E=64, k=6,
                   n_shared=2, bias="zipf", seed=4),
}


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32 holding them.

    Finite inputs only (the draws are Gaussian), so the uint32 sum cannot wrap."""
    u = np.array(a, dtype=np.float32, copy=True, order="C").view(np.uint32)
    u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    u &= np.uint32(0xFFFF0000)
    return u.view(np.float32)


def _normal(seed: int, tag: int, idx: int, shape, std: float) -> np.ndarray:
    rng = np.random.default_rng([seed, tag, idx])
    a = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    return round_to_bf16(a) if dtype == "bf16" else a.astype(np.float32)


def zipf_logit_bias(E: int, s: float = 1.1) -> np.ndarray:
    """Per-expert additive logit bias log p_e with p_e proportional to (e+1)^-s (input recipe of the Zipf-skewed E=64 workload)."""
    r = np.arange(1, E + 1, dtype=np.float64)
    p = r ** (-s)
    p /= p.sum()
    return np.log(p)[None, :].astype(np.float32)


@dataclasses.dataclass
class LayerInputs:
    cfg: LayerConfig
    x: np.ndarray            # [T, d]
    dy: Optional[np.ndarray]  # [T, d]
    w_router: np.ndarray     # [E, d]
    logit_bias: Optional[np.ndarray]  # [bias_groups, E] float32
    w_gate: np.ndarray       # [n_local + n_shared, f, d]
    w_up: np.ndarray         # [n_local + n_shared, f, d]
    w_down: np.ndarray       # [n_local + n_shared, d, f]


def make_inputs(cfg: LayerConfig, with_dy: Optional[bool] = None) -> LayerInputs:
    """Materialise every input tensor of one layer call (float32 arrays; bf16-exact for bf16 configs)."""
    T, d, f, E = cfg.T, cfg.d, cfg.f, cfg.E
    dt = cfg.dtype
    s = cfg.seed
    x = _store(_normal(s, TAG_X, 0, (T, d), 1.0), dt)
    if with_dy is None:
        with_dy = cfg.backward
    dy = _store(_normal(s, TAG_DY, 0, (T, d), 1.0), dt) if with_dy else None
    w_router = _store(_normal(s, TAG_WG, 0, (E, d), d ** -0.5), dt)
    bias = None
    if cfg.bias == "party":
        bias = _normal(s, TAG_BIAS, 0, (cfg.parties, E), 1.0)
    elif cfg.bias == "zipf":
        bias = zipf_logit_bias(E)
    elif cfg.bias == "forced_empty":
        bias = np.zeros((1, E), np.float32)
    G = cfg.n_groups
    w_gate = np.empty((G, f, d), np.float32)
    w_up = np.empty((G, f, d), np.float32)
    w_down = np.empty((G, d, f), np.float32)

    def fill(job):
        g, which = job
        if g < cfg.n_local:
            eid, tags = cfg.local_begin + g, (TAG_GATE, TAG_UP, TAG_DOWN)
        else:
            eid, tags = g - cfg.n_local, (TAG_SH_GATE, TAG_SH_UP, TAG_SH_DOWN)
        if which == 0:
            w_gate[g] = _store(_normal(s, tags[0], eid, (f, d), d ** -0.5), dt)
        elif which == 1:
            w_up[g] = _store(_normal(s, tags[1], eid, (f, d), d ** -0.5), dt)
        else:
            w_down[g] = _store(_normal(s, tags[2], eid, (d, f), f ** -0.5), dt)

    jobs = [(g, w) for g in range(G) for w in range(3)]
    workers = max(1, min(16, os.cpu_count() or 1, len(jobs)))
    with ThreadPoolExecutor(max_workers=workers) as ex:   # numpy's generators release the GIL
        list(ex.map(fill, jobs))
    return LayerInputs(cfg, x, dy, w_router, bias, w_gate, w_up, w_down)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bf16-exact (for host-side packing)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)

