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


def check_sampled(cfg, inp, layer, n_tokens=24, n_units=6, seed=0):
    """Full-size check: routing and permutation in full, every other output on samples the oracle
    computes one by one (tokens for y / dgate / dx, inner units for the weight gradients), and
    properties that hold at any size for the router's weight gradient."""
    tol = TOL[cfg.dtype]
    rng = np.random.default_rng(seed)
    L64 = O.router_logits(inp.x, inp.w_router, inp.logit_bias, cfg.bias_groups)
    L32 = O.selection_logits(L64)
    idx = O.topk_indices(L32, cfg.k)
    w = O.gate_weights(L64, idx, renormalize=cfg.renormalize)
    check_routing(cfg, layer, inp, L32, idx, w)
    counts, offsets, r2s, s2r = check_permutation(cfg, layer, inp, idx)
    errs = {}
    toks = np.unique(np.concatenate([[0, cfg.T - 1], rng.choice(cfg.T, n_tokens - 2, replace=False)]))
    tp = O.token_forward_backward(inp, toks, inp.dy[toks] if layer.backward_enabled else None)
    tt = torch.as_tensor(toks, device=layer.y.device)
    errs["y"] = assert_close("y[sampled]", np64(layer.y[tt]), tp["y"], tol)
    rows = s2r.reshape(cfg.T, cfg.k)[toks]
    sel = rows[rows >= 0]
    xp = layer.x_perm[torch.from_numpy(sel.astype(np.int64)).cuda()].float().cpu().numpy()
    assert np.array_equal(xp, inp.x[r2s[sel] // cfg.k].astype(np.float32)), "x_perm rows differ"
    if not layer.backward_enabled:
        return errs
    errs["dgate"] = assert_close("dgate[sampled]", layer.dgate.cpu().numpy()[toks], tp["dgate"], tol)
    dx_ref = tp["dx_experts"]
    if layer.router_backward:
        dL = O.router_logit_grad(L64[toks], idx[toks], w[toks], tp["dgate"], cfg.renormalize)
        errs["dlogits"] = assert_close("dlogits[sampled]", layer.dlogits.cpu().numpy()[toks], dL, tol)
        dx_ref = dx_ref + dL @ inp.w_router.astype(np.float64)
        # properties at full size: dW_router = dlogits^T x exactly as a sum, and its rows sum to zero
        gdl = layer.dlogits.cpu().numpy().astype(np.float64)
        gdw = layer.dw_router.cpu().numpy().astype(np.float64)
        errs["dW_router=dlogits^T x"] = assert_close("dW_router vs dlogits^T x", gdw, gdl.T @ inp.x.astype(np.float64),
                                                     1e-4)
        scale = np.abs(gdl).T @ np.abs(inp.x.astype(np.float64))
        assert np.max(np.abs(gdw.sum(axis=0))) <= 1e-3 * max(scale.max(), 1e-30) + 1e-6
    errs["dx"] = assert_close("dx[sampled]", np64(layer.dx[tt]), dx_ref, tol)
    # weight gradients on inner units of: heaviest, lightest non-empty, any empty, and shared experts
    dwg, dwu, dwd = layer.dw_gate, layer.dw_up, layer.dw_down
    groups = []
    if cfg.n_local:
        nz = np.nonzero(counts)[0]
        groups += [int(np.argmax(counts))]
        if len(nz):
            groups.append(int(nz[np.argmin(counts[nz])]))
        empty = np.nonzero(counts == 0)[0]
        for g in empty[:2]:
            assert not dwg[int(g)].any() and not dwu[int(g)].any() and not dwd[int(g)].any(), f"empty {g} dW"
    groups += [cfg.n_local + s for s in range(cfg.n_shared)]
    worst = 0.0
    for g in sorted(set(groups)):
        if g < cfg.n_local:
            rr = r2s[offsets[g]:offsets[g + 1]]
            tok = rr // cfg.k
            h = inp.x[tok]
            dO = w.reshape(-1)[rr][:, None] * inp.dy[tok].astype(np.float64)
        else:
            h, dO = inp.x, inp.dy
        units = np.sort(rng.choice(cfg.f, n_units, replace=False))
        ut = torch.as_tensor(units, device=dwg.device)
        sl = O.expert_wgrad_slices(h, dO, inp.w_gate[g], inp.w_up[g], inp.w_down[g], units, units)
        worst = max(worst, assert_close(f"dW_gate[{g}] rows", np64(dwg[g][ut]), sl["dW_gate_rows"], tol),
                    assert_close(f"dW_up[{g}] rows", np64(dwu[g][ut]), sl["dW_up_rows"], tol),
                    assert_close(f"dW_down[{g}] cols", np64(dwd[g][:, ut]), sl["dW_down_cols"], tol))
    errs["dW"] = worst
    return errs
