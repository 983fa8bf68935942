"""CPU oracle of the PC-MoE expert layer — TEST INFRASTRUCTURE, not part of the product.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import this module.
It shares no code with the HIP library (no headers, tables or helpers) and never imports it.

Plain, slow and fp64. Every function follows the paper's statement of the layer:

* Gating, Alg. 7 (Gating function): scores W_i h, p = softmax, I_e = TopKIndices(p), w_e = p[I_e].
  This layer renormalises w over the k selected experts (the workload's definition); the
  paper-literal unnormalised variant is kept behind ``renormalize=False``.
* Dispatch and combine, Alg. 3 (ProcessExperts): each selected expert receives the token's
  hidden state, runs ForwardExpert, and the owner forms sum_idx w_e[idx] * h^e_idx.
* Expert passes, Alg. 6 (ForwardExpert / BackwardExpert): h^e = E_j(h); backprop through E_j.
  Each expert is a SwiGLU feed-forward block W_down (silu(W_gate h) * (W_up h)).
* Backward, Alg. 5 (BackwardExperts) and Sec. 3.2 (backward propagation): the host of an
  expert receives the gradient w.r.t. that expert's output and returns the gradient w.r.t.
  its input; the router (part of the owner's backbone) is differentiated by the data owner.
* Expert sharding, Sec. 3.1 (2): a party hosts a shard of the global expert pool; here a
  contiguous range [local_begin, local_begin + local_count) of global expert ids.

Readings where the paper is silent (all listed in the design notes of the repository):
selection is taken on the float32 rounding of the fp64 logits (the kernel's precision) while
the gate weights are formed from the fp64 logits,
slot order within a token is descending logit with ties to the lower expert index, the
permutation is a stable counting sort of slots a = t*k + j by expert, and shared experts
(the footnote of Sec. 3.1: non-routed experts belong to the local model) are always active
with weight 1.
"""
from __future__ import annotations

import numpy as np


def f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------------------- gating (Alg. 7)

def router_logits(x, w_router, logit_bias=None, bias_groups=1):
    """Scores W_i h of the gating network (Alg. 7), plus an additive per-token-group bias.

    Token t uses bias row t // (T / bias_groups). Returns the fp64 values."""
    x, w = f64(x), f64(w_router)
    L = x @ w.T
    if logit_bias is not None:
        T = x.shape[0]
        group = np.arange(T) // (T // bias_groups)
        L = L + f64(logit_bias)[group]
    return L


def selection_logits(logits64):
    """The float32 values the top-k decision is taken on (the kernel's precision)."""
    return np.asarray(logits64, dtype=np.float64).astype(np.float32)


def topk_indices(logits, k):
    """TopKIndices of Alg. 7: the k largest scores per token, in descending order of score.

    Equal scores are ordered by the lower expert index (a stable sort of the negated scores;
    -0.0 and +0.0 compare equal)."""
    L = np.asarray(logits)
    order = np.argsort(-L, axis=1, kind="stable")
    return order[:, :k].astype(np.int32)


def softmax(L):
    L = f64(L)
    m = L.max(axis=1, keepdims=True)
    e = np.exp(L - m)
    return e / e.sum(axis=1, keepdims=True)


def gate_weights(logits, idx, renormalize=True):
    """w_e = p[I_e] with p = softmax of the scores (Alg. 7); optionally renormalised over I_e."""
    p = softmax(logits)
    w = np.take_along_axis(p, np.asarray(idx, dtype=np.int64), axis=1)
    if renormalize:
        w = w / w.sum(axis=1, keepdims=True)
    return w


# ------------------------------------------------------------------ dispatch (Alg. 3: hidden states to the experts' hosts)

def permutation(idx, local_begin, local_count):
    """Group the assignment slots a = t*k + j of the hosted experts by expert.

    Returns counts[local_count], offsets[local_count+1] (exclusive prefix sums),
    row_to_slot[N_loc] (slots in (expert, a) order: a stable sort) and slot_to_row[T*k]
    (its inverse, -1 for a slot whose expert is hosted elsewhere)."""
    idx = np.asarray(idx, dtype=np.int64)
    e_a = idx.reshape(-1)
    local = (e_a >= local_begin) & (e_a < local_begin + local_count)
    slots = np.nonzero(local)[0]
    counts = np.bincount(e_a[slots] - local_begin, minlength=local_count).astype(np.int32)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    row_to_slot = slots[np.argsort(e_a[slots], kind="stable")].astype(np.int32)
    slot_to_row = np.full(e_a.shape[0], -1, dtype=np.int32)
    slot_to_row[row_to_slot] = np.arange(row_to_slot.shape[0], dtype=np.int32)
    return counts, offsets, row_to_slot, slot_to_row


# --------------------------------------------------------------------- expert (Alg. 6, SwiGLU)

def silu(z):
    return z / (1.0 + np.exp(-z))


def dsilu(z):
    s = 1.0 / (1.0 + np.exp(-z))
    return s * (1.0 + z * (1.0 - s))


def expert_forward(h, w_gate, w_up, w_down):
    """ForwardExpert of Alg. 6 for one expert on a block of rows: returns G, U, Hid, O."""
    h = f64(h)
    G = h @ f64(w_gate).T
    U = h @ f64(w_up).T
    Hid = silu(G) * U
    O = Hid @ f64(w_down).T
    return G, U, Hid, O


def expert_backward(h, w_gate, w_up, w_down, G, U, Hid, dO):
    """BackwardExpert of Alg. 6: gradients of one expert given dL/d(expert output)."""
    h, w_gate, w_up, w_down, dO = f64(h), f64(w_gate), f64(w_up), f64(w_down), f64(dO)
    dHid = dO @ w_down
    dW_down = dO.T @ Hid
    dU = dHid * silu(G)
    dG = dHid * U * dsilu(G)
    dW_gate = dG.T @ h
    dW_up = dU.T @ h
    dh = dG @ w_gate + dU @ w_up
    return dict(dHid=dHid, dG=dG, dU=dU, dW_gate=dW_gate, dW_up=dW_up, dW_down=dW_down, dh=dh)


# ------------------------------------------------------------------------------ whole layer

def layer_forward(inp, *, renormalize=None):
    """The expert layer's forward pass for one party's shard (Alg. 3 with the gating of Alg. 7).

    ``inp`` holds x, w_router, logit_bias, w_gate, w_up, w_down and ``cfg`` (T, d, f, E, k,
    local_begin, n_local, n_shared, bias_groups, renormalize)."""
    cfg = inp.cfg
    ren = cfg.renormalize if renormalize is None else renormalize
    T, k = cfg.T, cfg.k
    Eloc, S = cfg.n_local, cfg.n_shared
    x = f64(inp.x)
    L64 = router_logits(x, inp.w_router, inp.logit_bias, cfg.bias_groups)
    L32 = selection_logits(L64)
    idx = topk_indices(L32, k)
    w = gate_weights(L64, idx, renormalize=ren)
    counts, offsets, row_to_slot, slot_to_row = permutation(idx, cfg.local_begin, Eloc)
    xp = x[row_to_slot // k]
    N = row_to_slot.shape[0]
    f, d = cfg.f, cfg.d
    G = np.zeros((N, f)); U = np.zeros((N, f)); Hid = np.zeros((N, f)); O = np.zeros((N, d))
    for e in range(Eloc):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            G[r0:r1], U[r0:r1], Hid[r0:r1], O[r0:r1] = expert_forward(
                xp[r0:r1], inp.w_gate[e], inp.w_up[e], inp.w_down[e])
    sh = [expert_forward(x, inp.w_gate[Eloc + s], inp.w_up[Eloc + s], inp.w_down[Eloc + s]) for s in range(S)]
    # owner-side combine of Alg. 3: sum over the token's selected (hosted) experts of w * output
    Y = np.zeros((T, d))
    for j in range(k):
        rows = slot_to_row[np.arange(T) * k + j]
        m = rows >= 0
        Y[m] += w[m, j:j + 1] * O[rows[m]]
    for s in range(S):
        Y += sh[s][3]
    return dict(logits64=L64, logits=L32, topk_idx=idx, topk_w=w, counts=counts, offsets=offsets,
                row_to_slot=row_to_slot, slot_to_row=slot_to_row, xp=xp, G=G, U=U, H=Hid, O=O,
                shared=sh, y=Y, renormalize=ren)


def layer_backward(inp, fwd, dy):
    """Backward of the layer (Alg. 5 + Alg. 6 + the adjoint of Alg. 7's gating).

    The host of an expert receives dL/d(expert output) = w * dY (the combine's adjoint) and
    returns dL/d(expert input); the router's gradient is formed on the data owner from the
    gate-weight gradients dgate[t, j] = <dY_t, O_row(t, j)>."""
    cfg = inp.cfg
    T, k, d, f = cfg.T, cfg.k, cfg.d, cfg.f
    Eloc, S = cfg.n_local, cfg.n_shared
    dy = f64(dy)
    x = f64(inp.x)
    w, O, slot_to_row, offsets = fwd["topk_w"], fwd["O"], fwd["slot_to_row"], fwd["offsets"]
    N = O.shape[0]
    # combine adjoint: dO_row = w * dY_t ; dgate = <dY_t, O_row>
    dO = np.zeros((N, d))
    dgate = np.zeros((T, k))
    for j in range(k):
        rows = slot_to_row[np.arange(T) * k + j]
        m = rows >= 0
        dO[rows[m]] = w[m, j:j + 1] * dy[m]
        dgate[m, j] = np.einsum("td,td->t", dy[m], O[rows[m]])
    dG = np.zeros((N, f)); dU = np.zeros((N, f)); dxp = np.zeros((N, d))
    G3 = (cfg.n_groups, f, d)
    dW_gate = np.zeros(G3); dW_up = np.zeros(G3); dW_down = np.zeros((cfg.n_groups, d, f))
    for e in range(Eloc):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            b = expert_backward(fwd["xp"][r0:r1], inp.w_gate[e], inp.w_up[e], inp.w_down[e],
                                fwd["G"][r0:r1], fwd["U"][r0:r1], fwd["H"][r0:r1], dO[r0:r1])
            dG[r0:r1], dU[r0:r1], dxp[r0:r1] = b["dG"], b["dU"], b["dh"]
            dW_gate[e], dW_up[e], dW_down[e] = b["dW_gate"], b["dW_up"], b["dW_down"]
    dx = np.zeros((T, d))
    for j in range(k):
        rows = slot_to_row[np.arange(T) * k + j]
        m = rows >= 0
        dx[m] += dxp[rows[m]]
    sh_b = []
    for s in range(S):
        Gs, Us, Hs, _ = fwd["shared"][s]
        b = expert_backward(x, inp.w_gate[Eloc + s], inp.w_up[Eloc + s], inp.w_down[Eloc + s], Gs, Us, Hs, dy)
        dW_gate[Eloc + s], dW_up[Eloc + s], dW_down[Eloc + s] = b["dW_gate"], b["dW_up"], b["dW_down"]
        dx += b["dh"]
        sh_b.append(b)
    out = dict(dO=dO, dgate=dgate, dG=dG, dU=dU, dxp=dxp, dW_gate=dW_gate, dW_up=dW_up, dW_down=dW_down,
               shared=sh_b, dx_experts=dx.copy())
    if cfg.router_backward:
        dL = router_logit_grad(fwd["logits64"], fwd["topk_idx"], w, dgate, fwd["renormalize"])
        dW_g = dL.T @ x
        dx = dx + dL @ f64(inp.w_router)
        out.update(dlogits=dL, dW_router=dW_g)
    out["dx"] = dx
    return out


def router_logit_grad(logits, idx, w, dgate, renormalize=True):
    """Adjoint of Alg. 7's gating: dL/dscores given dL/dw.

    Renormalised: w_j = exp(s_j) / sum_{j'} exp(s_{j'}) over the selected scores, so
    dscore[S_j] = w_j (dgate_j - sum_{j'} w_{j'} dgate_{j'}) and 0 off the selected set.
    Unnormalised (paper-literal): w_j = p[S_j] with p the softmax over all E scores, so
    dscore_e = p_e (g_e - sum_{e'} p_{e'} g_{e'}) with g the dgate scattered onto E.
    The selection itself is piecewise constant and contributes no gradient."""
    T, E = logits.shape
    idx = np.asarray(idx, dtype=np.int64)
    w, dgate = f64(w), f64(dgate)
    dL = np.zeros((T, E))
    if renormalize:
        s = (w * dgate).sum(axis=1, keepdims=True)
        np.put_along_axis(dL, idx, w * (dgate - s), axis=1)
    else:
        p = softmax(logits)
        g = np.zeros((T, E))
        np.put_along_axis(g, idx, dgate, axis=1)
        dL = p * (g - (p * g).sum(axis=1, keepdims=True))
    return dL


# ------------------------------------------------------ the whole layer one expert group at a time

def layer_streamed(inp, dy=None):
    """The same layer as layer_forward + layer_backward (Alg. 7, Alg. 3, Alg. 6, Alg. 5 and the router adjoint),
    evaluated one expert group at a time so that no array spans the whole row space: for large shapes whose
    per-row intermediates (G, U, H and their gradients over every routed row) do not fit in host memory at once.

    A generator. It yields, in this order:
      ("routing", dict(logits64, logits, topk_idx, topk_w, counts, offsets, row_to_slot, slot_to_row));
      ("group", g, dict(rows, tokens, O, and with dy: dO, dxp, dW_gate, dW_up, dW_down)) for every hosted
        routed expert g < n_local with at least one row (rows = its row-space indices, tokens = their tokens),
        then every shared expert (rows T*k + s*T + t for all tokens t);
      ("tokens", dict(y, and with dy: dgate, dx_experts, dx, and with the router adjoint: dlogits, dW_router)).
    Each group's forward and backward are those of expert_forward / expert_backward on its rows; the token
    outputs accumulate the groups' contributions (the owner-side combine of Alg. 3 and its adjoint)."""
    cfg = inp.cfg
    T, k, d = cfg.T, cfg.k, cfg.d
    Eloc, S = cfg.n_local, cfg.n_shared
    x = f64(inp.x)
    L64 = router_logits(x, inp.w_router, inp.logit_bias, cfg.bias_groups)
    L32 = selection_logits(L64)
    idx = topk_indices(L32, k)
    w = gate_weights(L64, idx, renormalize=cfg.renormalize)
    counts, offsets, row_to_slot, slot_to_row = permutation(idx, cfg.local_begin, Eloc)
    yield ("routing", dict(logits64=L64, logits=L32, topk_idx=idx, topk_w=w, counts=counts, offsets=offsets,
                           row_to_slot=row_to_slot, slot_to_row=slot_to_row))
    dyv = None if dy is None else f64(dy)
    wflat = w.reshape(-1)
    Y = np.zeros((T, d))
    dgate = np.zeros((T, k))
    dx = np.zeros((T, d))
    for g in range(Eloc + S):
        if g < Eloc:
            rows = np.arange(offsets[g], offsets[g + 1])
            if rows.size == 0:
                continue
            slots = row_to_slot[rows]
            tokens = slots // k
            wj = wflat[slots][:, None]                # gate weight of each row's slot
        else:
            s = g - Eloc
            tokens = np.arange(T)
            rows = T * k + s * T + tokens
            slots = None
            wj = np.ones((T, 1))                      # shared experts: always active, weight 1
        h = x[tokens]
        G, U, Hid, O = expert_forward(h, inp.w_gate[g], inp.w_up[g], inp.w_down[g])
        Y[tokens] += wj * O                           # a token meets each expert at most once
        out = dict(rows=rows, tokens=tokens, O=O)
        if dyv is not None:
            dO = wj * dyv[tokens]
            b = expert_backward(h, inp.w_gate[g], inp.w_up[g], inp.w_down[g], G, U, Hid, dO)
            dx[tokens] += b["dh"]
            if slots is not None:
                dgate[tokens, slots % k] = np.einsum("td,td->t", dyv[tokens], O)
            out.update(dO=dO, dxp=b["dh"], dW_gate=b["dW_gate"], dW_up=b["dW_up"], dW_down=b["dW_down"])
        yield ("group", g, out)
    tok = dict(y=Y)
    if dyv is not None:
        tok.update(dgate=dgate, dx_experts=dx.copy())
        if cfg.router_backward:
            dL = router_logit_grad(L64, idx, w, dgate, cfg.renormalize)
            tok.update(dlogits=dL, dW_router=dL.T @ x)
            dx = dx + dL @ f64(inp.w_router)
        tok["dx"] = dx
    yield ("tokens", tok)
