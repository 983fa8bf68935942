"""Pure-Python loop version of the expert layer for tiny shapes — test infrastructure only.

Written independently of moe_layer.py (no numpy linear algebra, no shared helpers): every
sum is an explicit loop over the definition, so the two agree only if both follow it.
Alg. 7 gating (renormalised over the selected experts), Alg. 3 dispatch/combine, Alg. 6
SwiGLU experts; shared experts always active with weight 1 (Sec. 3.1 footnote).
"""
import math


def _dot(a, b):
    s = 0.0
    for u, v in zip(a, b):
        s += u * v
    return s


def _ffn(h, wg, wu, wd):
    f = len(wg)
    hid = []
    for i in range(f):
        g = _dot(h, wg[i])
        u = _dot(h, wu[i])
        hid.append(g / (1.0 + math.exp(-g)) * u)
    return [_dot(hid, row) for row in wd]


def layer_forward(x, w_router, bias_rows, bias_groups, w_gate, w_up, w_down, k, local_begin, n_local,
                  n_shared, renormalize=True):
    """Returns (y, topk_idx, topk_w, counts, row_to_slot) using lists of floats only."""
    T = len(x)
    E = len(w_router)
    y = []
    all_idx, all_w = [], []
    for t in range(T):
        scores = []
        for e in range(E):
            s = _dot(x[t], w_router[e])
            if bias_rows is not None:
                s += bias_rows[t // (T // bias_groups)][e]
            scores.append(s)
        # selection: repeatedly take the largest remaining score, lower index on ties
        chosen = []
        for _ in range(k):
            best = None
            for e in range(E):
                if e in chosen:
                    continue
                if best is None or scores[e] > scores[best]:
                    best = e
            chosen.append(best)
        mx = max(scores)
        z_all = sum(math.exp(s - mx) for s in scores)
        p_sel = [math.exp(scores[e] - mx) / z_all for e in chosen]
        if renormalize:
            z = sum(p_sel)
            p_sel = [p / z for p in p_sel]
        all_idx.append(chosen)
        all_w.append(p_sel)
        out = [0.0] * len(x[t])
        for j, e in enumerate(chosen):
            g = e - local_begin
            if 0 <= g < n_local:
                o = _ffn(x[t], w_gate[g], w_up[g], w_down[g])
                out = [a + p_sel[j] * b for a, b in zip(out, o)]
        for s in range(n_shared):
            g = n_local + s
            o = _ffn(x[t], w_gate[g], w_up[g], w_down[g])
            out = [a + b for a, b in zip(out, o)]
        y.append(out)
    counts = [0] * n_local
    row_to_slot = []
    for g in range(n_local):
        for t in range(T):
            for j in range(k):
                if all_idx[t][j] == local_begin + g:
                    counts[g] += 1
                    row_to_slot.append(t * k + j)
    return y, all_idx, all_w, counts, row_to_slot
