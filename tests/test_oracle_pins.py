"""Pins of the CPU oracle against things other than itself.

Each pin is a function taking the oracle module, so the planted-mistake tests at the end can
run it on a deliberately broken copy of the oracle and show that it fails.

* finite differences of <dY, Y> on tiny shapes (the whole backward, Alg. 5/6 and the
  adjoint of Alg. 7's gating);
* a dense reformulation with torch's library silu/softmax and autograd (forward and backward
  through a one-hot combine instead of a permutation);
* a pure-loop brute force (selection, gate weights, permutation order, forward);
* closed forms: E=1/k=1 is one dense expert; k=E renormalised is the full softmax; all-zero
  router gives experts 0..k-1 with weight 1/k; duplicated router rows tie to the lower index;
* invariants: gate weights sum to 1 and are non-increasing, counts sum to T*k, the
  permutation is a bijection with ascending slots per expert, identical experts make Y
  independent of routing, Euler identities of the 1-homogeneous expert weights, shard
  outputs sum to the full layer.
"""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.special import softmax as sp_softmax, expit

from oracle import moe_layer, brute
from paper_2506_02965_amd.synth import LayerConfig, LayerInputs, make_inputs


# ------------------------------------------------------------------------------- helpers

def tiny_inputs(seed, T=6, d=4, f=5, E=4, k=2, n_shared=0, local_begin=0, local_count=None, bias=False,
                bias_groups=1, renormalize=True, router_backward=True, min_gap=1e-3):
    """fp64 random layer whose top-(k+1) score gaps all exceed min_gap (no selection flips under FD)."""
    cfg = LayerConfig("tiny", T=T, d=d, f=f, E=E, k=k, n_shared=n_shared, local_begin=local_begin,
                      local_count=local_count, dtype="f32", renormalize=renormalize,
                      router_backward=router_backward, bias="party" if bias else None,
                      parties=bias_groups)
    for s in range(seed, seed + 1000):
        rng = np.random.default_rng([s, 77])
        G = cfg.n_groups
        inp = LayerInputs(
            cfg,
            x=rng.standard_normal((T, d)),
            dy=rng.standard_normal((T, d)),
            w_router=rng.standard_normal((E, d)),
            logit_bias=rng.standard_normal((bias_groups, E)) if bias else None,
            w_gate=rng.standard_normal((G, f, d)) / np.sqrt(d),
            w_up=rng.standard_normal((G, f, d)) / np.sqrt(d),
            w_down=rng.standard_normal((G, d, f)) / np.sqrt(f),
        )
        L = moe_layer.router_logits(inp.x, inp.w_router, inp.logit_bias, cfg.bias_groups)
        Ls = -np.sort(-L, axis=1)[:, :min(k + 1, E)]
        if Ls.shape[1] < 2 or np.min(-np.diff(Ls, axis=1)) > min_gap:
            return inp
    raise RuntimeError("no well-separated draw")


def loss_of(ml, inp):
    return float((ml.layer_forward(inp)["y"] * inp.dy).sum())


def fd_grad(ml, inp, name, h=1e-6):
    a = getattr(inp, name)
    g = np.zeros_like(a)
    it = np.nditer(a, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        old = a[i]
        a[i] = old + h
        lp = loss_of(ml, inp)
        a[i] = old - h
        lm = loss_of(ml, inp)
        a[i] = old
        g[i] = (lp - lm) / (2 * h)
    return g


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ---------------------------------------------------------------------------------- pins

def pin_finite_differences(ml, **kw):
    inp = tiny_inputs(1, **kw)
    fwd = ml.layer_forward(inp)
    bwd = ml.layer_backward(inp, fwd, inp.dy)
    checks = {"w_gate": bwd["dW_gate"], "w_up": bwd["dW_up"], "w_down": bwd["dW_down"]}
    if inp.cfg.router_backward:
        # a party shard leaves the router term of dX to the data owner, so only full layers check x here
        checks["x"] = bwd["dx"]
        checks["w_router"] = bwd["dW_router"]
    for name, an in checks.items():
        num = fd_grad(ml, inp, name)
        assert rel(an, num) < 1e-6, (name, rel(an, num))


def dense_torch(inp, router_grad=True):
    """The same layer written densely: coefficient C[t,e] = sum_j [idx_tj = e] w_tj, no permutation."""
    cfg = inp.cfg
    tt = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    x, wr, wg, wu, wd = tt(inp.x), tt(inp.w_router), tt(inp.w_gate), tt(inp.w_up), tt(inp.w_down)
    L = x @ wr.T
    if inp.logit_bias is not None:
        grp = torch.arange(cfg.T) // (cfg.T // cfg.bias_groups)
        L = L + torch.tensor(np.asarray(inp.logit_bias, np.float64))[grp]
    # the decision itself is piecewise constant: take it on float32 scores with a stable sort
    idx = torch.from_numpy(np.argsort(-L.detach().numpy().astype(np.float32), axis=1, kind="stable")[:, :cfg.k].copy())
    p = torch.softmax(L if router_grad else L.detach(), dim=1)
    w = p.gather(1, idx)
    if cfg.renormalize:
        w = w / w.sum(dim=1, keepdim=True)
    C = torch.zeros(cfg.T, cfg.E, dtype=torch.float64).scatter_add(1, idx, w)
    Y = torch.zeros(cfg.T, cfg.d, dtype=torch.float64)
    for g in range(cfg.n_local):
        e = cfg.local_begin + g
        out = F.linear(F.silu(F.linear(x, wg[g])) * F.linear(x, wu[g]), wd[g])
        Y = Y + C[:, e:e + 1] * out
    for s in range(cfg.n_shared):
        g = cfg.n_local + s
        Y = Y + F.linear(F.silu(F.linear(x, wg[g])) * F.linear(x, wu[g]), wd[g])
    (Y * torch.tensor(np.asarray(inp.dy, np.float64))).sum().backward()
    return dict(y=Y.detach().numpy(), dx=x.grad.numpy(),
                dW_router=None if wr.grad is None else wr.grad.numpy(), dW_gate=wg.grad.numpy(),
                dW_up=wu.grad.numpy(), dW_down=wd.grad.numpy(), idx=idx.numpy(), w=w.detach().numpy())


def pin_dense_torch(ml, **kw):
    inp = tiny_inputs(3, T=16, d=8, f=12, E=6, k=3, **kw)
    fwd = ml.layer_forward(inp)
    bwd = ml.layer_backward(inp, fwd, inp.dy)
    ref = dense_torch(inp, router_grad=inp.cfg.router_backward)
    assert np.array_equal(fwd["topk_idx"], ref["idx"])
    assert rel(fwd["topk_w"], ref["w"]) < 1e-12
    assert rel(fwd["y"], ref["y"]) < 1e-12
    for nm in ("dW_gate", "dW_up", "dW_down"):
        assert rel(bwd[nm], ref[nm]) < 1e-11, nm
    assert rel(bwd["dx"], ref["dx"]) < 1e-11
    if inp.cfg.router_backward:
        assert rel(bwd["dW_router"], ref["dW_router"]) < 1e-11


def pin_brute_force(ml, **kw):
    inp = tiny_inputs(5, T=10, d=6, f=7, E=5, k=2, **kw)
    cfg = inp.cfg
    fwd = ml.layer_forward(inp)
    lst = lambda a: np.asarray(a).tolist()
    y, idx, w, counts, r2s = brute.layer_forward(
        lst(inp.x), lst(inp.w_router), None if inp.logit_bias is None else lst(inp.logit_bias), cfg.bias_groups,
        lst(inp.w_gate), lst(inp.w_up), lst(inp.w_down), cfg.k, cfg.local_begin, cfg.n_local, cfg.n_shared,
        cfg.renormalize)
    assert np.array_equal(fwd["topk_idx"], np.array(idx))
    assert rel(fwd["topk_w"], w) < 1e-12
    assert np.array_equal(fwd["counts"], np.array(counts))
    assert np.array_equal(fwd["row_to_slot"], np.array(r2s, dtype=np.int32))
    assert rel(fwd["y"], y) < 1e-12


def pin_gate_invariants(ml):
    inp = make_inputs(LayerConfig("g", T=256, d=64, f=64, E=16, k=4, dtype="f32", seed=11))
    fwd = ml.layer_forward(inp)
    w = fwd["topk_w"]
    assert np.max(np.abs(w.sum(axis=1) - 1.0)) < 1e-14
    assert np.all(np.diff(w, axis=1) <= 1e-15)           # non-increasing in slot j
    L = fwd["logits"]
    sel = np.take_along_axis(L, fwd["topk_idx"].astype(np.int64), axis=1)
    assert np.all(np.diff(sel, axis=1) <= 0)               # descending scores
    kth = sel[:, -1:]
    others = L.copy()
    np.put_along_axis(others, fwd["topk_idx"].astype(np.int64), -np.inf, axis=1)
    assert np.all(others <= kth)                            # nothing unselected beats the k-th


def pin_full_softmax(ml):
    """k = E with renormalisation: the gate weights are the full softmax, in sorted order."""
    rng = np.random.default_rng(4)
    L = rng.standard_normal((50, 7))
    idx = ml.topk_indices(L.astype(np.float32), 7)
    w = ml.gate_weights(L, idx, renormalize=True)
    ref = np.take_along_axis(sp_softmax(L, axis=1), idx.astype(np.int64), axis=1)
    assert rel(w, ref) < 1e-14
    # unnormalised weights are the softmax probabilities of the selected experts
    w2 = ml.gate_weights(L, idx[:, :2], renormalize=False)
    assert rel(w2, np.take_along_axis(sp_softmax(L, axis=1), idx[:, :2].astype(np.int64), axis=1)) < 1e-14


def pin_ties(ml):
    # all scores equal: experts 0..k-1 in index order, weight 1/k
    L = np.zeros((5, 8), np.float32)
    idx = ml.topk_indices(L, 3)
    assert np.array_equal(idx, np.tile(np.arange(3), (5, 1)))
    assert rel(ml.gate_weights(L, idx), np.full((5, 3), 1 / 3)) < 1e-15
    # -0.0 and +0.0 are equal scores
    L2 = np.array([[0.0, -0.0, 1.0, -0.0]], np.float32)
    L2[0, 0] = -0.0
    assert ml.topk_indices(L2, 3).tolist() == [[2, 0, 1]]
    # duplicated router rows: exact ties resolve to the lower index
    rng = np.random.default_rng(9)
    x = rng.standard_normal((40, 8))
    wr = rng.standard_normal((6, 8))
    wr[4] = wr[1]
    idx = ml.topk_indices(ml.selection_logits(ml.router_logits(x, wr)), 6)
    pos = {e: np.argmax(idx == e, axis=1) for e in (1, 4)}
    assert np.all(pos[1] < pos[4])


def pin_permutation(ml):
    rng = np.random.default_rng(2)
    T, k, E = 300, 3, 9
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    for lb, lc in ((0, E), (2, 4), (8, 1)):
        counts, offsets, r2s, s2r = ml.permutation(idx, lb, lc)
        e_a = idx.reshape(-1)
        local = (e_a >= lb) & (e_a < lb + lc)
        assert counts.sum() == local.sum() and offsets[-1] == local.sum()
        if lc == E:
            assert counts.sum() == T * k
        # brute force: for each expert in order, its slots in increasing order
        ref = [a for e in range(lb, lb + lc) for a in range(T * k) if e_a[a] == e]
        assert r2s.tolist() == ref
        assert np.all(s2r[r2s] == np.arange(len(r2s)))
        assert np.all(s2r[~local] == -1)
        for g in range(lc):
            seg = r2s[offsets[g]:offsets[g + 1]]
            assert np.all(e_a[seg] == lb + g) and np.all(np.diff(seg) > 0)


def pin_dense_expert(ml):
    """E = 1, k = 1: every token goes to the single expert with weight 1; Y is that expert's FFN."""
    rng = np.random.default_rng(21)
    T, d, f = 33, 8, 12
    cfg = LayerConfig("e1", T=T, d=d, f=f, E=1, k=1, dtype="f32")
    inp = LayerInputs(cfg, rng.standard_normal((T, d)), rng.standard_normal((T, d)), rng.standard_normal((1, d)),
                      None, rng.standard_normal((1, f, d)), rng.standard_normal((1, f, d)),
                      rng.standard_normal((1, d, f)))
    fwd = ml.layer_forward(inp)
    gate = inp.x @ inp.w_gate[0].T
    dense = (gate * expit(gate) * (inp.x @ inp.w_up[0].T)) @ inp.w_down[0].T   # Swish_1(xW) * xV, then W2
    assert np.all(fwd["topk_w"] == 1.0)
    assert fwd["row_to_slot"].tolist() == list(range(T))
    assert rel(fwd["y"], dense) < 1e-13
    bwd = ml.layer_backward(inp, fwd, inp.dy)
    assert np.all(bwd["dW_router"] == 0)    # k = 1 renormalised: the gate weight is constantly 1


def pin_hand_worked(ml):
    """A two-token layer small enough to work out by hand (d = 2, E = 2, k = 1, f = 1, integer weights).

    Token 0 = (1, 0) scores (2, 0) and goes to expert 0; token 1 = (0, 1) scores (0, 1) and goes to expert 1, each
    with gate weight 1 (top-1, renormalised). With s1 = sigmoid(1), s2 = sigmoid(2):
      expert 0: G = 1, U = 1, H = s1,          O = W_down0 H = ( s1, -s1)
      expert 1: G = 2, U = 3, H = 2 s2 * 3,     O = W_down1 H = (2H, H)
    Backward with dY = I: dO = dY rows; dH = W_down^T dO = 1 for both tokens;
      dU = dH silu(G), dG = dH U s(G) (1 + G (1 - s(G)));
      dx0 = (dG0 + dU0, dU0), dx1 = (0, 2 dG1 + 3 dU1); dW_down_e = dO_e H_e, dW_gate_e = dG_e x_e,
      dW_up_e = dU_e x_e; dgate_t = <dY_t, O_t>; the router gradient is 0 (the weight is constantly 1)."""
    import math
    s1, s2 = 1 / (1 + math.exp(-1.0)), 1 / (1 + math.exp(-2.0))
    cfg = LayerConfig("hand", T=2, d=2, f=1, E=2, k=1, dtype="f32")
    inp = LayerInputs(cfg, x=np.array([[1.0, 0.0], [0.0, 1.0]]), dy=np.eye(2),
                      w_router=np.array([[2.0, 0.0], [0.0, 1.0]]), logit_bias=None,
                      w_gate=np.array([[[1.0, 0.0]], [[0.0, 2.0]]]), w_up=np.array([[[1.0, 1.0]], [[0.0, 3.0]]]),
                      w_down=np.array([[[1.0], [-1.0]], [[2.0], [1.0]]]))
    H0, H1 = s1, 2 * s2 * 3
    dU0, dG0 = s1, 1 * s1 * (1 + (1 - s1))
    dU1, dG1 = 2 * s2, 3 * s2 * (1 + 2 * (1 - s2))
    fwd = ml.layer_forward(inp)
    assert fwd["topk_idx"].reshape(-1).tolist() == [0, 1]
    assert np.allclose(fwd["topk_w"].reshape(-1), [1.0, 1.0], rtol=0, atol=1e-15)
    assert np.allclose(fwd["y"], [[H0, -H0], [2 * H1, H1]], rtol=1e-14, atol=0)
    bwd = ml.layer_backward(inp, fwd, inp.dy)
    assert np.allclose(bwd["dgate"].reshape(-1), [H0, H1], rtol=1e-14, atol=0)
    assert np.allclose(bwd["dx"], [[dG0 + dU0, dU0], [0.0, 2 * dG1 + 3 * dU1]], rtol=1e-14, atol=1e-15)
    assert np.allclose(bwd["dW_down"], [[[H0], [0.0]], [[0.0], [H1]]], rtol=1e-14, atol=1e-15)
    assert np.allclose(bwd["dW_gate"], [[[dG0, 0.0]], [[0.0, dG1]]], rtol=1e-14, atol=1e-15)
    assert np.allclose(bwd["dW_up"], [[[dU0, 0.0]], [[0.0, dU1]]], rtol=1e-14, atol=1e-15)
    assert np.all(bwd["dW_router"] == 0)


def pin_identical_experts(ml):
    """All routed experts share weights: renormalised gate weights sum to 1, so Y = FFN(x)."""
    cfg = LayerConfig("ident", T=64, d=16, f=24, E=6, k=3, dtype="f32", seed=5)
    inp = make_inputs(cfg)
    for a in (inp.w_gate, inp.w_up, inp.w_down):
        a[:] = a[0]
    fwd = ml.layer_forward(inp)
    G, U, H, O = ml.expert_forward(inp.x, inp.w_gate[0], inp.w_up[0], inp.w_down[0])
    assert rel(fwd["y"], O) < 1e-13
    assert len(set(fwd["topk_idx"].reshape(-1).tolist())) > 1


def pin_euler_identities(ml):
    """O_e is 1-homogeneous in W_up_e and in W_down_e: <dW, W>_F = <dO_e, O_e>_F for both."""
    cfg = LayerConfig("euler", T=96, d=16, f=24, E=4, k=2, n_shared=1, dtype="f32", seed=8)
    inp = make_inputs(cfg, with_dy=True)
    fwd = ml.layer_forward(inp)
    bwd = ml.layer_backward(inp, fwd, inp.dy)
    for e in range(cfg.n_local):
        r0, r1 = fwd["offsets"][e], fwd["offsets"][e + 1]
        ip = float((bwd["dO"][r0:r1] * fwd["O"][r0:r1]).sum())
        assert abs(float((bwd["dW_up"][e] * inp.w_up[e]).sum()) - ip) < 1e-10 * max(1, abs(ip))
        assert abs(float((bwd["dW_down"][e] * inp.w_down[e]).sum()) - ip) < 1e-10 * max(1, abs(ip))
    # combine adjoint: sum_j w_tj dgate_tj = <dY_t, Y_routed_t>
    y_routed = fwd["y"] - fwd["shared"][0][3]
    lhs = (fwd["topk_w"] * bwd["dgate"]).sum(axis=1)
    assert rel(lhs, (inp.dy * y_routed).sum(axis=1)) < 1e-12
    # router adjoint: every row of dscores sums to zero (softmax is shift invariant)
    assert np.max(np.abs(bwd["dlogits"].sum(axis=1))) < 1e-12


def pin_shards_sum_to_layer(ml):
    """Four disjoint expert shards (Sec. 3.1 (2)): partial outputs add up to the full layer."""
    base = LayerConfig("shard", T=64, d=16, f=24, E=8, k=3, dtype="f32", bias="party", parties=4, seed=13)
    full_inp = make_inputs(base, with_dy=True)
    full = ml.layer_forward(full_inp)
    fb = ml.layer_backward(full_inp, full, full_inp.dy)
    y = np.zeros_like(full["y"]); dxe = np.zeros_like(full["y"]); dgate = np.zeros_like(fb["dgate"])
    for p in range(4):
        cfg = dataclasses.replace(base, local_begin=2 * p, local_count=2, router_backward=False)
        inp = dataclasses.replace(full_inp, cfg=cfg, w_gate=full_inp.w_gate[2 * p:2 * p + 2],
                                  w_up=full_inp.w_up[2 * p:2 * p + 2], w_down=full_inp.w_down[2 * p:2 * p + 2])
        fw = ml.layer_forward(inp)
        bw = ml.layer_backward(inp, fw, inp.dy)
        assert np.array_equal(fw["topk_idx"], full["topk_idx"])
        y += fw["y"]; dxe += bw["dx"]; dgate += bw["dgate"]
        for g in range(2):
            assert rel(bw["dW_gate"][g], fb["dW_gate"][2 * p + g]) < 1e-12
    assert rel(y, full["y"]) < 1e-12
    assert rel(dxe, fb["dx_experts"]) < 1e-12
    assert rel(dgate, fb["dgate"]) < 1e-12


# ---------------------------------------------------------------------------- the tests

@pytest.mark.parametrize("kw", [
    dict(),
    dict(n_shared=1),
    dict(renormalize=False),
    dict(bias=True, bias_groups=2),
    dict(E=4, k=4),
    dict(local_begin=1, local_count=2, router_backward=False),
])
def test_finite_differences(kw):
    pin_finite_differences(moe_layer, **kw)


@pytest.mark.parametrize("kw", [dict(), dict(n_shared=2), dict(renormalize=False), dict(bias=True, bias_groups=4),
                                dict(local_begin=2, local_count=3, router_backward=False)])
def test_dense_torch(kw):
    pin_dense_torch(moe_layer, **kw)


@pytest.mark.parametrize("kw", [dict(), dict(n_shared=1), dict(renormalize=False),
                                dict(local_begin=1, local_count=3)])
def test_brute_force(kw):
    pin_brute_force(moe_layer, **kw)


def test_gate_invariants():
    pin_gate_invariants(moe_layer)


def test_full_softmax():
    pin_full_softmax(moe_layer)


def test_ties():
    pin_ties(moe_layer)


def test_permutation():
    pin_permutation(moe_layer)


def test_dense_expert():
    pin_dense_expert(moe_layer)


def test_hand_worked():
    pin_hand_worked(moe_layer)


def test_identical_experts():
    pin_identical_experts(moe_layer)


def test_euler_identities():
    pin_euler_identities(moe_layer)


def test_shards_sum_to_layer():
    pin_shards_sum_to_layer(moe_layer)


def _streamed(inp):
    out = {"groups": {}}
    for item in moe_layer.layer_streamed(inp, inp.dy):
        if item[0] == "group":
            out["groups"][item[1]] = item[2]
        else:
            out[item[0]] = item[1]
    return out


@pytest.mark.parametrize("kw", [
    dict(T=48, d=16, f=24, E=8, k=3, n_shared=1, bias="zipf", seed=17),            # router adjoint + shared
    dict(T=64, d=16, f=24, E=8, k=2, local_begin=2, local_count=4, router_backward=False, bias="party",
         parties=4, seed=18),                                                          # a party's shard
    dict(T=40, d=8, f=16, E=4, k=2, renormalize=False, seed=19),                       # paper-literal gating
])
def test_layer_streamed_matches_layer(kw):
    """The one-group-at-a-time evaluation used for the largest shapes gives every output of the whole-layer
    oracle: routing and permutation exactly, the row-space rows of each group, each expert's weight gradients,
    and the token outputs."""
    cfg = LayerConfig("stream", dtype="f32", **kw)
    inp = make_inputs(cfg, with_dy=True)
    fwd = moe_layer.layer_forward(inp)
    bwd = moe_layer.layer_backward(inp, fwd, inp.dy)
    st = _streamed(inp)
    for key in ("topk_idx", "counts", "offsets", "row_to_slot", "slot_to_row"):
        assert np.array_equal(st["routing"][key], fwd[key]), key
    assert np.array_equal(st["routing"]["topk_w"], fwd["topk_w"])
    N, TK = len(fwd["row_to_slot"]), cfg.T * cfg.k
    seen = []
    for g, grp in st["groups"].items():
        rows = grp["rows"]
        if g < cfg.n_local:
            assert rows.min() >= 0 and rows.max() < N
            assert rel(grp["O"], fwd["O"][rows]) < 1e-12
            assert rel(grp["dO"], bwd["dO"][rows]) < 1e-12
            assert rel(grp["dxp"], bwd["dxp"][rows]) < 1e-12
        else:
            s = g - cfg.n_local
            assert np.array_equal(rows, TK + s * cfg.T + np.arange(cfg.T))
            assert rel(grp["O"], fwd["shared"][s][3]) < 1e-12
            assert rel(grp["dxp"], bwd["shared"][s]["dh"]) < 1e-12
        for wname in ("dW_gate", "dW_up", "dW_down"):
            assert rel(grp[wname], bwd[wname][g]) < 1e-12, (g, wname)
        seen.append(g)
    # every group with rows is visited once, empty hosted experts are not
    want = [g for g in range(cfg.n_local) if fwd["counts"][g]] + list(range(cfg.n_local, cfg.n_groups))
    assert seen == want
    tok = st["tokens"]
    assert rel(tok["y"], fwd["y"]) < 1e-12
    assert rel(tok["dgate"], bwd["dgate"]) < 1e-12
    assert rel(tok["dx"], bwd["dx"]) < 1e-12
    if cfg.router_backward:
        assert rel(tok["dlogits"], bwd["dlogits"]) < 1e-12
        assert rel(tok["dW_router"], bwd["dW_router"]) < 1e-12
    else:
        assert "dlogits" not in tok


# ----------------------------------------------- planted mistakes: each pin catches its kind

def _fails(pin, *a, **kw):
    try:
        pin(*a, **kw)
    except AssertionError:
        return True
    return False


def test_planted_wrong_silu_derivative(monkeypatch):
    monkeypatch.setattr(moe_layer, "dsilu", lambda z: expit(z))          # drops the z*s*(1-s) term
    assert _fails(pin_finite_differences, moe_layer)
    assert _fails(pin_dense_torch, moe_layer)
    assert _fails(pin_hand_worked, moe_layer)


def test_planted_silu_on_up_projection(monkeypatch):
    def bad_forward(h, w_gate, w_up, w_down):
        G = h @ w_gate.T
        U = h @ w_up.T
        Hid = G * moe_layer.silu(U)
        return G, U, Hid, Hid @ w_down.T
    monkeypatch.setattr(moe_layer, "expert_forward", bad_forward)
    assert _fails(pin_dense_torch, moe_layer)
    assert _fails(pin_brute_force, moe_layer)
    assert _fails(pin_hand_worked, moe_layer)


def test_planted_missing_renormalisation(monkeypatch):
    orig = moe_layer.gate_weights
    monkeypatch.setattr(moe_layer, "gate_weights", lambda L, idx, renormalize=True: orig(L, idx, False))
    assert _fails(pin_gate_invariants, moe_layer)
    assert _fails(pin_identical_experts, moe_layer)


def test_planted_tie_to_higher_index(monkeypatch):
    def bad_topk(L, k):
        L = np.asarray(L)
        E = L.shape[1]
        order = E - 1 - np.argsort(-L[:, ::-1], axis=1, kind="stable")
        return order[:, :k].astype(np.int32)
    monkeypatch.setattr(moe_layer, "topk_indices", bad_topk)
    assert _fails(pin_ties, moe_layer)


def test_planted_unstable_permutation(monkeypatch):
    orig = moe_layer.permutation

    def bad_perm(idx, lb, lc):
        counts, offsets, r2s, s2r = orig(idx, lb, lc)
        for g in range(lc):
            r2s[offsets[g]:offsets[g + 1]] = r2s[offsets[g]:offsets[g + 1]][::-1]
        s2r[:] = -1
        s2r[r2s] = np.arange(len(r2s))
        return counts, offsets, r2s, s2r
    monkeypatch.setattr(moe_layer, "permutation", bad_perm)
    assert _fails(pin_permutation, moe_layer)
    assert _fails(pin_brute_force, moe_layer)


def test_planted_router_gradient_sign(monkeypatch):
    orig = moe_layer.router_logit_grad
    monkeypatch.setattr(moe_layer, "router_logit_grad", lambda *a, **k: -orig(*a, **k))
    assert _fails(pin_finite_differences, moe_layer)
    assert _fails(pin_dense_torch, moe_layer)


def test_planted_transposed_down_projection(monkeypatch):
    orig = moe_layer.expert_backward

    def bad_backward(h, w_gate, w_up, w_down, G, U, Hid, dO):
        out = orig(h, w_gate, w_up, w_down, G, U, Hid, dO)
        out["dW_down"] = out["dW_down"] * 0.5
        return out
    monkeypatch.setattr(moe_layer, "expert_backward", bad_backward)
    assert _fails(pin_finite_differences, moe_layer)
    assert _fails(pin_euler_identities, moe_layer)
    assert _fails(pin_hand_worked, moe_layer)
