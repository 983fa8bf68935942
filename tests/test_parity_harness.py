"""CPU checks of the GPU parity harness itself (tests/gpu_util.py): fed the oracle's own outputs, rounded to the
storage precision as the GPU stores them, both comparisons pass; a planted error in any one output tensor, in
one row or one expert, makes them fail. No GPU is touched: the "layer" holds CPU tensors."""
import types

import numpy as np
import pytest
import torch

from oracle import moe_layer as O
from paper_2506_02965_amd.synth import LayerConfig, make_inputs
from gpu_util import check_full, check_full_streamed


def fake_layer(cfg, inp):
    """The outputs a correct layer would produce, from the whole-layer oracle, in the GPU's storage dtypes."""
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    fwd = O.layer_forward(inp)
    bwd = O.layer_backward(inp, fwd, inp.dy)
    T, k, d, S = cfg.T, cfg.k, cfg.d, cfg.n_shared
    N, TK, R = len(fwd["row_to_slot"]), T * k, T * k + S * T
    st = lambda a: torch.as_tensor(np.asarray(a, np.float64)).to(dt)
    f32 = lambda a: torch.as_tensor(np.asarray(a, np.float32))
    i32 = lambda a: torch.as_tensor(np.asarray(a, np.int32))
    L = types.SimpleNamespace(backward_enabled=True, router_backward=cfg.router_backward)
    L.logits, L.topk_idx, L.topk_w = f32(fwd["logits"]), i32(fwd["topk_idx"]), f32(fwd["topk_w"])
    L.counts, L.offsets = i32(fwd["counts"]), i32(fwd["offsets"])
    r2s = np.full(TK, -1, np.int32)
    r2s[:N] = fwd["row_to_slot"]
    L.row_to_slot, L.slot_to_row = i32(r2s), i32(fwd["slot_to_row"])
    xp = np.zeros((TK, d))
    xp[:N] = inp.x[fwd["row_to_slot"] // k]
    L.x_perm = st(xp)
    yp, dyp, dxp = np.zeros((R, d)), np.zeros((TK, d)), np.zeros((R, d))
    yp[:N], dyp[:N], dxp[:N] = fwd["O"], bwd["dO"], bwd["dxp"]
    for s in range(S):
        yp[TK + s * T:TK + (s + 1) * T] = fwd["shared"][s][3]
        dxp[TK + s * T:TK + (s + 1) * T] = bwd["shared"][s]["dh"]
    L.y_perm, L.dy_perm, L.dx_perm, L.y, L.dx = st(yp), st(dyp), st(dxp), st(fwd["y"]), st(bwd["dx"])
    L.dgate = f32(bwd["dgate"])
    L.dw_gate, L.dw_up, L.dw_down = st(bwd["dW_gate"]), st(bwd["dW_up"]), st(bwd["dW_down"])
    if cfg.router_backward:
        L.dlogits, L.dw_router = f32(bwd["dlogits"]), f32(bwd["dW_router"])
    return L


CASES = {
    "shared_zipf": LayerConfig("h1", T=96, d=128, f=128, E=8, k=3, n_shared=1, bias="zipf", seed=41),
    "shard": LayerConfig("h2", T=128, d=128, f=128, E=8, k=2, local_begin=2, local_count=4,
                         router_backward=False, bias="party", parties=4, seed=42),
}


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("check", [check_full, check_full_streamed], ids=["whole", "streamed"])
def test_harness_accepts_the_oracle(name, check):
    cfg = CASES[name]
    inp = make_inputs(cfg, with_dy=True)
    errs = check(cfg, inp, fake_layer(cfg, inp))
    assert max(errs.values()) < 1e-2


def _plant(L, attr, where):
    t = getattr(L, attr)
    t[where] = t[where] * 1.5 + 1.0


@pytest.mark.parametrize("attr,where", [
    ("dx_perm", (5, slice(None))),          # one routed row of the input gradient
    ("y_perm", (7, slice(0, 8))),           # part of one routed output row
    ("dw_down", (1, 3, slice(None))),       # one row of one expert's weight gradient
    ("dw_gate", (0, slice(None), 2)),       # one column of another expert's
    ("dy", (11, slice(None))),              # one token of the layer's input gradient
    ("dgate", (3, 1)),                      # one gate gradient
    ("dw_router", (2, slice(None))),        # one router row
    ("topk_idx", (4, 0)),                   # routing
])
@pytest.mark.parametrize("check", [check_full, check_full_streamed], ids=["whole", "streamed"])
def test_harness_catches_a_planted_error(attr, where, check):
    cfg = CASES["shared_zipf"]
    inp = make_inputs(cfg, with_dy=True)
    L = fake_layer(cfg, inp)
    if attr == "dy":
        attr = "dx"
    if attr == "topk_idx":
        L.topk_idx[where] = (L.topk_idx[where] + 1) % cfg.E
    else:
        _plant(L, attr, where)
    with pytest.raises(AssertionError):
        check(cfg, inp, L)
