"""One MoE expert layer on the GPU: torch owns the buffers, libpcmoe computes every step.

Forward (Alg. 3 with the gating of Alg. 7 and the experts of Alg. 6):
    moe_route -> moe_permute -> moe_expert_ffn_fwd -> moe_combine
Backward (Alg. 5 / Alg. 6 and the owner-side router adjoint):
    moe_combine_bwd -> moe_expert_ffn_bwd -> moe_route_bwd (full layer only) -> moe_permute_bwd
Expert update (the last step of Alg. 6): moe_expert_update over the hosted experts' weights.
All calls are enqueued on one stream; no per-expert count ever returns to the host.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from . import pcmoe as P


@dataclass
class LayerWeights:
    x: torch.Tensor
    w_router: torch.Tensor
    logit_bias: Optional[torch.Tensor]
    bias_groups: int
    w_gate: torch.Tensor
    w_up: torch.Tensor
    w_down: torch.Tensor
    dy: Optional[torch.Tensor] = None


def torch_dtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def upload(inp, device="cuda") -> LayerWeights:
    """Copy a synth.LayerInputs (float32 arrays, bf16-exact for bf16 layers) to the device."""
    cfg = inp.cfg
    dt = torch_dtype(cfg.dtype)
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device=device).to(dt)
    bias = None
    if inp.logit_bias is not None:
        bias = torch.from_numpy(np.ascontiguousarray(inp.logit_bias, dtype=np.float32)).to(device)
    return LayerWeights(to(inp.x), to(inp.w_router), bias, cfg.bias_groups, to(inp.w_gate), to(inp.w_up),
                        to(inp.w_down), None if inp.dy is None else to(inp.dy))


class MoELayer:
    def __init__(self, cfg, device="cuda", backward=None, router_backward=None):
        self.cfg = cfg
        self.device = device
        self.backward_enabled = cfg.backward if backward is None else backward
        self.router_backward = cfg.router_backward if router_backward is None else router_backward
        self.desc = P.make_desc(cfg.T, cfg.d, cfg.f, cfg.E, cfg.k, cfg.local_begin, cfg.n_local, cfg.n_shared,
                                cfg.renormalize, cfg.dtype)
        T, d, f, E, k, S, Eloc = cfg.T, cfg.d, cfg.f, cfg.E, cfg.k, cfg.n_shared, cfg.n_local
        dt = torch_dtype(cfg.dtype)
        R = T * k + S * T
        kw = dict(device=device)
        self.logits = torch.empty(T, E, dtype=torch.float32, **kw)
        self.topk_idx = torch.empty(T, k, dtype=torch.int32, **kw)
        self.topk_w = torch.empty(T, k, dtype=torch.float32, **kw)
        self.counts = torch.empty(max(Eloc, 1), dtype=torch.int32, **kw)
        self.offsets = torch.empty(Eloc + 1, dtype=torch.int32, **kw)
        self.row_to_slot = torch.empty(T * k, dtype=torch.int32, **kw)
        self.slot_to_row = torch.empty(T * k, dtype=torch.int32, **kw)
        self.x_perm = torch.empty(T * k, d, dtype=dt, **kw)
        self.y_perm = torch.empty(R, d, dtype=dt, **kw)
        self.y = torch.empty(T, d, dtype=dt, **kw)
        ws = lambda which: torch.empty(max(P.moe_workspace_size(self.desc, which), 1), dtype=torch.uint8, **kw)
        self.ws_permute = ws(P.MOE_WS_PERMUTE)
        self.saved = ws(P.MOE_WS_FFN_SAVED)
        self.ws_ffn_fwd = ws(P.MOE_WS_FFN_FWD)
        if self.backward_enabled:
            G = Eloc + S
            self.dy_perm = torch.empty(T * k, d, dtype=dt, **kw)
            self.dgate = torch.empty(T, k, dtype=torch.float32, **kw)
            self.dx_perm = torch.empty(R, d, dtype=dt, **kw)
            self.dw_gate = torch.empty(G, f, d, dtype=dt, **kw)
            self.dw_up = torch.empty(G, f, d, dtype=dt, **kw)
            self.dw_down = torch.empty(G, d, f, dtype=dt, **kw)
            self.ws_ffn_bwd = ws(P.MOE_WS_FFN_BWD)
            self.dx = torch.empty(T, d, dtype=dt, **kw)
            if self.router_backward:
                self.dlogits = torch.empty(T, E, dtype=torch.float32, **kw)
                self.dw_router = torch.empty(E, d, dtype=torch.float32, **kw)
                self.ws_route_bwd = ws(P.MOE_WS_ROUTE_BWD)

    # ------------------------------------------------------------------ forward
    def route(self, w: LayerWeights):
        P.moe_route(self.desc, w.x, w.w_router, w.logit_bias, w.bias_groups, self.logits, self.topk_idx, self.topk_w)

    def permute(self, w: LayerWeights):
        P.moe_permute(self.desc, self.topk_idx, w.x, self.counts, self.offsets, self.row_to_slot, self.slot_to_row,
                      self.x_perm, self.ws_permute, self.ws_permute.numel())

    def ffn_fwd(self, w: LayerWeights):
        P.moe_expert_ffn_fwd(self.desc, w.x, self.x_perm, self.offsets, w.w_gate, w.w_up, w.w_down, self.y_perm,
                             self.saved, self.ws_ffn_fwd, self.ws_ffn_fwd.numel())

    def combine(self):
        P.moe_combine(self.desc, self.y_perm, self.slot_to_row, self.topk_w, self.y)

    def forward(self, w: LayerWeights):
        self.route(w)
        self.permute(w)
        self.ffn_fwd(w)
        self.combine()
        return self.y

    # ----------------------------------------------------------------- backward
    def combine_bwd(self, dy):
        P.moe_combine_bwd(self.desc, dy, self.y_perm, self.slot_to_row, self.topk_w, self.dy_perm, self.dgate)

    def ffn_bwd(self, w: LayerWeights, dy):
        P.moe_expert_ffn_bwd(self.desc, w.x, self.x_perm, dy, self.dy_perm, self.offsets, w.w_gate, w.w_up, w.w_down,
                             self.saved, self.dx_perm, self.dw_gate, self.dw_up, self.dw_down, self.ws_ffn_bwd,
                             self.ws_ffn_bwd.numel())

    def route_bwd(self, w: LayerWeights):
        P.moe_route_bwd(self.desc, w.x, self.logits, self.topk_idx, self.topk_w, self.dgate, self.dlogits,
                        self.dw_router, self.ws_route_bwd, self.ws_route_bwd.numel())

    def permute_bwd(self, w: LayerWeights):
        P.moe_permute_bwd(self.desc, self.dx_perm, self.slot_to_row, self.dlogits if self.router_backward else None,
                          w.w_router, self.dx)

    def backward(self, w: LayerWeights, dy=None):
        dy = w.dy if dy is None else dy
        self.combine_bwd(dy)
        self.ffn_bwd(w, dy)
        if self.router_backward:
            self.route_bwd(w)
        self.permute_bwd(w)
        return self.dx

    # ------------------------------------------------------------- expert update
    def init_update_state(self, w: LayerWeights, master: bool = True):
        """fp32 optimiser state over w_gate, w_up, w_down (in that order): zero moments and, if asked,
        a master copy of the current weights."""
        n = w.w_gate.numel() + w.w_up.numel() + w.w_down.numel()
        kw = dict(device=self.device, dtype=torch.float32)
        self.opt_m = torch.zeros(n, **kw)
        self.opt_v = torch.zeros(n, **kw)
        self.opt_master = None
        if master:  # filled slice by slice: no transient copy of all parameters
            self.opt_master = torch.empty(n, **kw)
            o = 0
            for t in (w.w_gate, w.w_up, w.w_down):
                self.opt_master[o:o + t.numel()].copy_(t.reshape(-1))
                o += t.numel()
        self.opt_step = 0

    def update(self, w: LayerWeights, opt: "P.moe_opt"):
        """One optimiser step of the hosted experts from the gradients of the last backward."""
        self.opt_step += 1
        opt.step = self.opt_step
        P.moe_expert_update(self.desc, opt, w.w_gate, w.w_up, w.w_down, self.dw_gate, self.dw_up, self.dw_down,
                            self.opt_master, self.opt_m, self.opt_v)

    def n_local_rows(self) -> int:
        return int(self.offsets[-1].item())


def training_footprint(cfg, local_count: int, master: bool = True) -> dict:
    """Device bytes one party allocates for the expert layer's training step (route, permute, expert FFN forward
    and backward, combine and its adjoint, router adjoint, expert AdamW update) when it hosts `local_count` of the
    cfg.E routed experts, by category:
      expert_state  hosted experts' weights and weight gradients (dtype) plus fp32 moments and master copy;
      activations   row-space buffers (capacity T*k + S*T rows), saved activations and the FFN workspaces;
      owner         the owner-side buffers of its own T tokens (input, router, combine, input gradient).
    The sizes are those MoELayer and init_update_state allocate, with workspace sizes from the library."""
    T, d, f, E, k, S = cfg.T, cfg.d, cfg.f, cfg.E, cfg.k, cfg.n_shared
    es = 2 if cfg.dtype == "bf16" else 4
    desc = P.make_desc(T, d, f, E, k, 0, local_count, S, cfg.renormalize, cfg.dtype)
    ws = lambda which: max(P.moe_workspace_size(desc, which), 1)
    G, R = local_count + S, T * k + S * T
    params = G * 3 * f * d
    expert_state = params * es * 2 + params * 4 * (3 if master else 2)
    activations = (T * k * d * es            # x_perm
                   + R * d * es              # y_perm
                   + T * k * d * es          # dy_perm
                   + R * d * es              # dx_perm
                   + ws(P.MOE_WS_FFN_SAVED) + ws(P.MOE_WS_FFN_FWD) + ws(P.MOE_WS_FFN_BWD) + ws(P.MOE_WS_PERMUTE)
                   + (local_count + 1) * 4 + max(local_count, 1) * 4 + 2 * T * k * 4)   # offsets, counts, maps
    owner = (T * d * es * 3                  # x, y, dx
             + T * d * es                    # dy
             + E * d * es + E * d * 4        # router weights and their gradient
             + T * E * 4 * 2                 # logits, dlogits
             + T * k * (4 + 4 + 4)           # topk_idx, topk_w, dgate
             + ws(P.MOE_WS_ROUTE_BWD))
    return {"local_experts": local_count, "expert_state": expert_state, "activations": activations, "owner": owner,
            "total": expert_state + activations + owner}
