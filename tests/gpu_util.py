"""Helpers of the GPU parity tests: run the HIP layer through the C ABI and compare with the oracle.

The bar: integer outputs (routing, permutation) bit-exact; floating outputs within a max relative
error max|got - ref| / max|ref| per tensor (each expert's weight gradient its own tensor) of 1e-4
for fp32 layers and 2e-2 for bf16 layers."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import moe_layer as O
from paper_2506_02965_amd.layer import MoELayer, upload

TOL = {"f32": 1e-4, "bf16": 2e-2}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def np64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def maxrel(got, ref):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    if den == 0.0:
        return float(np.max(np.abs(got))) if got.size else 0.0
    return float(np.max(np.abs(got - ref)) / den)


def assert_close(name, got, ref, tol):
    e = maxrel(got, ref)
    assert e <= tol, f"{name}: max relative error {e:.3e} > {tol:.0e}"
    return e


def run_gpu(cfg, inp, backward=None):
    torch.cuda.synchronize()
    w = upload(inp)
    layer = MoELayer(cfg, backward=backward)
    layer.forward(w)
    if layer.backward_enabled:
        layer.backward(w)
    torch.cuda.synchronize()
    return layer, w


def check_logits(gpu_logits, ref32):
    g = np.ascontiguousarray(gpu_logits.cpu().numpy()).view(np.int32).astype(np.int64)
    r = np.ascontiguousarray(ref32.astype(np.float32)).view(np.int32).astype(np.int64)
    ulp = np.abs(g - r)
    assert ulp.max() <= 1, f"logits differ by {ulp.max()} ulp"
    assert (ulp == 0).mean() >= 0.999, f"only {(ulp == 0).mean():.5f} of the logits are bit-identical"


def check_routing(cfg, layer, inp, ref_logits32, ref_idx, ref_w):
    check_logits(layer.logits, ref_logits32)
    assert np.array_equal(layer.topk_idx.cpu().numpy(), ref_idx), "topk_idx differs"
    assert_close("topk_w", layer.topk_w.cpu().numpy(), ref_w, 1e-5)


def check_permutation(cfg, layer, inp, ref_idx):
    counts, offsets, r2s, s2r = O.permutation(ref_idx, cfg.local_begin, cfg.n_local)
    assert np.array_equal(layer.counts.cpu().numpy()[:cfg.n_local], counts), "counts differ"
    assert np.array_equal(layer.offsets.cpu().numpy(), offsets), "offsets differ"
    g_r2s = layer.row_to_slot.cpu().numpy()
    n = len(r2s)
    assert np.array_equal(g_r2s[:n], r2s), "row_to_slot differs"
    assert np.all(g_r2s[n:] == -1), "row_to_slot tail is not -1"
    assert np.array_equal(layer.slot_to_row.cpu().numpy(), s2r), "slot_to_row differs"
    return counts, offsets, r2s, s2r


def check_full(cfg, inp, layer):
    """Element-by-element comparison of every output with the whole-layer oracle."""
    tol = TOL[cfg.dtype]
    fwd = O.layer_forward(inp)
    check_routing(cfg, layer, inp, fwd["logits"], fwd["topk_idx"], fwd["topk_w"])
    counts, offsets, r2s, s2r = check_permutation(cfg, layer, inp, fwd["topk_idx"])
    N = len(r2s)
    xp = layer.x_perm[:N].float().cpu().numpy()
    assert np.array_equal(xp, inp.x[r2s // cfg.k].astype(np.float32)), "x_perm rows differ (a byte copy)"
    errs = {}
    errs["y"] = assert_close("y", np64(layer.y), fwd["y"], tol)
    errs["y_perm"] = assert_close("y_perm routed", np64(layer.y_perm[:N]), fwd["O"], tol) if N else 0.0
    TK = cfg.T * cfg.k
    for s in range(cfg.n_shared):
        errs[f"y_shared{s}"] = assert_close(f"y_perm shared {s}", np64(layer.y_perm[TK + s * cfg.T:TK + (s + 1) * cfg.T]),
                                            fwd["shared"][s][3], tol)
    if not layer.backward_enabled:
        return errs
    bwd = O.layer_backward(inp, fwd, inp.dy)
    errs["dgate"] = assert_close("dgate", layer.dgate.cpu().numpy(), bwd["dgate"], tol)
    if N:
        errs["dy_perm"] = assert_close("dy_perm", np64(layer.dy_perm[:N]), bwd["dO"], tol)
        errs["dx_perm"] = assert_close("dx_perm", np64(layer.dx_perm[:N]), bwd["dxp"], tol)
    dwg, dwu, dwd = np64(layer.dw_gate), np64(layer.dw_up), np64(layer.dw_down)
    worst = 0.0
    for g in range(cfg.n_groups):
        if g < cfg.n_local and counts[g] == 0:
            assert not dwg[g].any() and not dwu[g].any() and not dwd[g].any(), f"empty expert {g}: dW not zero"
            continue
        worst = max(worst, assert_close(f"dW_gate[{g}]", dwg[g], bwd["dW_gate"][g], tol),
                    assert_close(f"dW_up[{g}]", dwu[g], bwd["dW_up"][g], tol),
                    assert_close(f"dW_down[{g}]", dwd[g], bwd["dW_down"][g], tol))
    errs["dW"] = worst
    if layer.router_backward:
        errs["dlogits"] = assert_close("dlogits", layer.dlogits.cpu().numpy(), bwd["dlogits"], tol)
        errs["dW_router"] = assert_close("dW_router", layer.dw_router.cpu().numpy(), bwd["dW_router"], tol)
    errs["dx"] = assert_close("dx", np64(layer.dx), bwd["dx"], tol)
    return errs


class RowSpaceErr:
    """max|got - ref| / max|ref| of one tensor compared block by block."""

    def __init__(self):
        self.diff = 0.0
        self.ref = 0.0

    def add(self, got, ref):
        got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
        if ref.size:
            self.diff = max(self.diff, float(np.max(np.abs(got - ref))))
            self.ref = max(self.ref, float(np.max(np.abs(ref))))

    def check(self, name, tol):
        e = self.diff / self.ref if self.ref > 0 else self.diff
        assert e <= tol, f"{name}: max relative error {e:.3e} > {tol:.0e}"
        return e


def check_full_streamed(cfg, inp, layer, log_every=1):
    """Element-by-element comparison of every output with the oracle evaluated one expert group at a time
    (oracle.moe_layer.layer_streamed): the same bar as check_full, for shapes whose whole-layer oracle arrays
    would not fit in host memory at once. Routing and permutation bit-exact; x_perm byte-exact; y_perm, dy_perm
    and dx_perm over all their rows; every group's dW_gate, dW_up and dW_down; y, dgate, dlogits, dW_router
    and dx over all tokens."""
    tol = TOL[cfg.dtype]
    errs = {}
    stream = O.layer_streamed(inp, inp.dy if layer.backward_enabled else None)
    kind, rt = next(stream)
    assert kind == "routing"
    check_routing(cfg, layer, inp, rt["logits"], rt["topk_idx"], rt["topk_w"])
    counts, offsets, r2s, s2r = check_permutation(cfg, layer, inp, rt["topk_idx"])
    N = len(r2s)
    for r0 in range(0, N, 16384):
        r1 = min(N, r0 + 16384)
        xp = layer.x_perm[r0:r1].float().cpu().numpy()
        assert np.array_equal(xp, inp.x[r2s[r0:r1] // cfg.k].astype(np.float32)), f"x_perm rows {r0}..{r1} differ"
    y_perm, dy_perm, dx_perm = RowSpaceErr(), RowSpaceErr(), RowSpaceErr()
    worst_dw = 0.0
    visited = set()
    for item in stream:
        if item[0] != "group":
            tok = item[1]
            break
        _, g, grp = item
        visited.add(g)
        rows = torch.as_tensor(grp["rows"], device=layer.y_perm.device)
        y_perm.add(np64(layer.y_perm[rows]), grp["O"])
        if layer.backward_enabled:
            if g < cfg.n_local:
                dy_perm.add(np64(layer.dy_perm[rows]), grp["dO"])
            dx_perm.add(np64(layer.dx_perm[rows]), grp["dxp"])
            worst_dw = max(worst_dw,
                           assert_close(f"dW_gate[{g}]", np64(layer.dw_gate[g]), grp["dW_gate"], tol),
                           assert_close(f"dW_up[{g}]", np64(layer.dw_up[g]), grp["dW_up"], tol),
                           assert_close(f"dW_down[{g}]", np64(layer.dw_down[g]), grp["dW_down"], tol))
        if log_every and len(visited) % log_every == 0:
            log(f"[parity]   group {g}: {len(grp['rows'])} rows checked")
    errs["y_perm"] = y_perm.check("y_perm", tol)
    errs["y"] = assert_close("y", np64(layer.y), tok["y"], tol)
    if not layer.backward_enabled:
        return errs
    # hosted experts without a row have exact-zero weight gradients
    for g in range(cfg.n_local):
        if counts[g] == 0:
            assert g not in visited
            assert not layer.dw_gate[g].any() and not layer.dw_up[g].any() and not layer.dw_down[g].any(), \
                f"empty expert {g}: dW not zero"
    errs["dy_perm"] = dy_perm.check("dy_perm", tol)
    errs["dx_perm"] = dx_perm.check("dx_perm", tol)
    errs["dW"] = worst_dw
    errs["dgate"] = assert_close("dgate", layer.dgate.cpu().numpy(), tok["dgate"], tol)
    if layer.router_backward:
        errs["dlogits"] = assert_close("dlogits", layer.dlogits.cpu().numpy(), tok["dlogits"], tol)
        errs["dW_router"] = assert_close("dW_router", layer.dw_router.cpu().numpy(), tok["dW_router"], tol)
    errs["dx"] = assert_close("dx", np64(layer.dx), tok["dx"], tol)
    return errs
