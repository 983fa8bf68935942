"""Oracle of the expert parameter update — test infrastructure, not part of the product.

Alg. 6 ends the host's expert step with an update of the expert's parameters and leaves the optimiser open.
Two are offered, each written from its definition, in fp64 over the exact stored values:

* SGD with weight decay added to the gradient: p <- p - lr * (g + wd * p).
* AdamW, Adam with decoupled weight decay (Loshchilov & Hutter, "Decoupled Weight Decay
  Regularization", ICLR 2019), in the order of its algorithm: decay the parameter, update the
  first and second moments, correct their bias for step t, take the step.

Only tests/, the smoke check and the benchmark's CPU baseline may import this module.
"""
from __future__ import annotations

import numpy as np


def sgd_step(p, g, lr, weight_decay):
    """One SGD step; returns the new parameters (fp64)."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64)
    return p - lr * (g + weight_decay * p)


def adamw_step(p, g, m, v, lr, beta1, beta2, eps, weight_decay, t):
    """One AdamW step at step number t >= 1; returns (p, m, v) as fp64 arrays."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64)
    m = np.asarray(m, np.float64)
    v = np.asarray(v, np.float64)
    p = p * (1.0 - lr * weight_decay)                 # decoupled weight decay
    m = beta1 * m + (1.0 - beta1) * g                 # first moment
    v = beta2 * v + (1.0 - beta2) * g * g             # second moment
    m_hat = m / (1.0 - beta1 ** t)                    # bias corrections
    v_hat = v / (1.0 - beta2 ** t)
    p = p - lr * m_hat / (np.sqrt(v_hat) + eps)
    return p, m, v


def expert_update(opt, weights, grads, master=None, m=None, v=None):
    """The whole update over a list of parameter arrays (w_gate, w_up, w_down) with their gradients.

    master, m and v are the flat fp32 state arrays in the order of `weights` (or None). Returns
    (new master or new weights in fp64, new m, new v), flat and in the same order."""
    src = np.concatenate([np.asarray(w, np.float64).ravel() for w in weights]) if master is None \
        else np.asarray(master, np.float64)
    g = np.concatenate([np.asarray(x, np.float64).ravel() for x in grads])
    if opt["kind"] == "sgd":
        return sgd_step(src, g, opt["lr"], opt["weight_decay"]), None, None
    return adamw_step(src, g, m, v, opt["lr"], opt["beta1"], opt["beta2"], opt["eps"], opt["weight_decay"],
                      opt["step"])
