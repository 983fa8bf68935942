"""Pins of the expert-update oracle (oracle/moe_update.py) against things other than itself:
PyTorch's own AdamW and SGD (library routines, fp64 on the CPU, several steps), the closed form of
AdamW's first step, and invariants. Planted mistakes in the oracle must fail a pin."""
import numpy as np
import pytest
import torch

from oracle import moe_update as U

OPT = dict(kind="adamw", lr=3e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


def _torch_adamw(p0, grads, o):
    p = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=o["lr"], betas=(o["beta1"], o["beta2"]), eps=o["eps"],
                            weight_decay=o["weight_decay"], foreach=False)
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    st = opt.state[p]
    return p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


def _oracle_adamw(p0, grads, o):
    p, m, v = p0.astype(np.float64), np.zeros_like(p0, np.float64), np.zeros_like(p0, np.float64)
    for t, g in enumerate(grads, start=1):
        p, m, v = U.adamw_step(p, g, m, v, o["lr"], o["beta1"], o["beta2"], o["eps"], o["weight_decay"], t)
    return p, m, v


def test_adamw_matches_torch_over_steps():
    rng = np.random.default_rng(0)
    p0 = rng.standard_normal(4096)
    grads = [rng.standard_normal(4096) * s for s in (1.0, 0.3, 2.0, 1e-3, 0.7)]
    want = _torch_adamw(p0, grads, OPT)
    got = _oracle_adamw(p0, grads, OPT)
    for a, b in zip(got, want):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-15)


def test_sgd_matches_torch():
    rng = np.random.default_rng(1)
    p0 = rng.standard_normal(1000)
    g = rng.standard_normal(1000)
    p = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.SGD([p], lr=0.05, weight_decay=0.01)
    p.grad = torch.tensor(g)
    opt.step()
    np.testing.assert_allclose(U.sgd_step(p0, g, 0.05, 0.01), p.detach().numpy(), rtol=1e-14)


def test_adamw_first_step_closed_form():
    # at t = 1 the corrected moments are g and g^2, so the step is lr * g / (|g| + eps)
    rng = np.random.default_rng(2)
    p0, g = rng.standard_normal(512), rng.standard_normal(512)
    lr, wd, eps = 1e-2, 0.05, 1e-8
    p, m, v = U.adamw_step(p0, g, np.zeros(512), np.zeros(512), lr, 0.9, 0.999, eps, wd, 1)
    np.testing.assert_allclose(p, p0 * (1 - lr * wd) - lr * g / (np.abs(g) + eps), rtol=1e-13)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-13)


def test_adamw_zero_gradient_fixed_point():
    p0 = np.linspace(-2, 2, 100)
    p, m, v = U.adamw_step(p0, np.zeros(100), np.zeros(100), np.zeros(100), 1e-3, 0.9, 0.999, 1e-8, 0.0, 7)
    assert np.array_equal(p, p0) and not m.any() and not v.any()


def test_expert_update_flattens_in_order():
    rng = np.random.default_rng(3)
    ws = [rng.standard_normal((2, 4, 8)) for _ in range(3)]
    gs = [rng.standard_normal((2, 4, 8)) for _ in range(3)]
    n = sum(w.size for w in ws)
    o = dict(OPT, step=1)
    p, m, v = U.expert_update(o, ws, gs, m=np.zeros(n), v=np.zeros(n))
    for i in range(3):
        pi, _, _ = U.adamw_step(ws[i].ravel(), gs[i].ravel(), np.zeros(64), np.zeros(64), o["lr"], o["beta1"],
                                o["beta2"], o["eps"], o["weight_decay"], 1)
        np.testing.assert_array_equal(p[64 * i:64 * (i + 1)], pi)


def _planted(monkeypatch, fn):
    monkeypatch.setattr(U, "adamw_step", fn)


def test_planted_missing_bias_correction_fails(monkeypatch):
    def wrong(p, g, m, v, lr, b1, b2, eps, wd, t):
        p = p * (1 - lr * wd)
        m = b1 * m + (1 - b1) * g
        v = b2 * v + (1 - b2) * g * g
        return p - lr * m / (np.sqrt(v) + eps), m, v
    _planted(monkeypatch, wrong)
    with pytest.raises(AssertionError):
        test_adamw_matches_torch_over_steps()


def test_planted_coupled_weight_decay_fails(monkeypatch):
    orig = U.adamw_step

    def wrong(p, g, m, v, lr, b1, b2, eps, wd, t):  # L2 decay folded into the gradient (Adam, not AdamW)
        return orig(p, np.asarray(g) + wd * np.asarray(p), m, v, lr, b1, b2, eps, 0.0, t)
    _planted(monkeypatch, wrong)
    with pytest.raises(AssertionError):
        test_adamw_matches_torch_over_steps()
