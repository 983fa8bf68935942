"""Parity of moe_expert_update (through the C ABI) with the update oracle on the GPU.

Small cases compare every element: the fp32 master copy, fp32 weights and the moments within the
fp32 bar (max |got - ref| / max |ref| per tensor <= 1e-4), the step itself (new - old parameters)
within 1e-3 of its own size, and bf16 weights against the oracle's result rounded to bf16 (within one
unit in the last place, nearly all exact). The config-2 expert shapes run in full in the launch
configuration the benchmark times and are compared on a random sample of parameters."""
import numpy as np
import pytest
import torch

from oracle import moe_update as U
from paper_2506_02965_amd import pcmoe as P
from paper_2506_02965_amd.synth import round_to_bf16
from gpu_util import TOL, assert_close, log

STEP_TOL = 1e-3  # the update (new - old) relative to its own largest magnitude

pytestmark = pytest.mark.gpu


def bf16_ulp_diff(a, b):
    """|a - b| in bf16 units of the last place (a, b: float32 arrays of bf16 values)."""
    ia = a.astype(np.float32).view(np.int32) >> 16
    ib = b.astype(np.float32).view(np.int32) >> 16
    # map the sign-magnitude bit patterns onto a monotone integer line
    ia = np.where(ia < 0, -(ia & 0x7fff), ia)
    ib = np.where(ib < 0, -(ib & 0x7fff), ib)
    return np.abs(ia.astype(np.int64) - ib.astype(np.int64))


def make_case(G, f, d, dtype, master, seed):
    rng = np.random.default_rng(seed)
    shapes = [(G, f, d), (G, f, d), (G, d, f)]
    m32 = [rng.standard_normal(s).astype(np.float32) * 0.05 for s in shapes]
    g32 = [(rng.standard_normal(s) * 0.01).astype(np.float32) for s in shapes]
    if dtype == "bf16":
        w32 = [round_to_bf16(x) for x in m32]
        g32 = [round_to_bf16(x) for x in g32]
    else:
        w32 = [x.copy() for x in m32]
    n = sum(int(np.prod(s)) for s in shapes)
    mom = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    vel = (rng.random(n) * 1e-4).astype(np.float32)
    return shapes, w32, g32, (np.concatenate([x.ravel() for x in m32]) if master else None), mom, vel


def run_case(G, f, d, dtype, master, kind, steps, seed):
    shapes, w32, g32, mst, mom, vel = make_case(G, f, d, dtype, master, seed)
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = lambda a, t=dt: torch.from_numpy(np.ascontiguousarray(a)).cuda().to(t)
    W = [dev(x) for x in w32]
    Gd = [dev(x) for x in g32]
    M = dev(mst, torch.float32) if mst is not None else None
    Mo, Ve = dev(mom, torch.float32), dev(vel, torch.float32)
    desc = P.make_desc(T=8, d_model=d, d_ff=f, n_experts=max(G, 2), top_k=1, local_count=G, dtype=dtype)
    exp_src = mst.astype(np.float64) if mst is not None else np.concatenate([x.ravel() for x in w32]).astype(np.float64)
    exp_m, exp_v = mom.astype(np.float64), vel.astype(np.float64)
    o = dict(kind=kind, lr=2e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    for t in range(1, steps + 1):
        opt = P.make_opt(kind=kind, lr=o["lr"], beta1=o["beta1"], beta2=o["beta2"], eps=o["eps"],
                         weight_decay=o["weight_decay"], step=t)
        log(f"update {dtype} master={master} {kind} G={G} f={f} d={d} step {t}")
        P.moe_expert_update(desc, opt, W[0], W[1], W[2], Gd[0], Gd[1], Gd[2], M, Mo if kind == "adamw" else None,
                            Ve if kind == "adamw" else None)
        torch.cuda.synchronize()
        # the oracle steps from the state the kernel stepped from: fp32 values (master or the dtype weights)
        prev = exp_src
        res, nm, nv = U.expert_update(dict(o, step=t), [], g32, master=exp_src, m=exp_m, v=exp_v)
        if kind == "adamw":
            exp_m, exp_v = nm, nv
        exp_src = res if mst is not None else np.concatenate(
            [x.float().cpu().numpy().ravel() for x in W]).astype(np.float64)
        got_w = np.concatenate([x.float().cpu().numpy().ravel() for x in W])
        want_w = round_to_bf16(res.astype(np.float32)) if dtype == "bf16" else res
        if dtype == "bf16":
            ulp = bf16_ulp_diff(got_w, want_w.astype(np.float32))
            assert ulp.max() <= 1 and (ulp == 0).mean() > 0.99, (ulp.max(), (ulp == 0).mean())
        else:
            assert_close("weights", got_w, want_w, TOL["f32"])
            assert_close("weight step", got_w - prev, want_w - prev, STEP_TOL)
        if M is not None:
            got = M.cpu().numpy().astype(np.float64)
            assert_close("master", got, res, TOL["f32"])
            assert_close("master step", got - prev, res - prev, STEP_TOL)
            exp_src = got   # continue from the kernel's fp32 state, as it does
        if kind == "adamw":
            for name, got_t, want in (("m", Mo, exp_m), ("v", Ve, exp_v)):
                assert_close(name, got_t.cpu().numpy(), want, TOL["f32"])
            exp_m, exp_v = Mo.cpu().numpy().astype(np.float64), Ve.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("dtype,master,kind", [
    ("bf16", True, "adamw"), ("bf16", False, "adamw"), ("f32", False, "adamw"),
    ("bf16", True, "sgd"), ("f32", False, "sgd"),
])
def test_update_small(dtype, master, kind):
    run_case(G=3, f=256, d=128, dtype=dtype, master=master, kind=kind, steps=3, seed=40)


def test_update_zero_gradient_fixed_point():
    """g = 0, no decay, zero moments: AdamW leaves every parameter bit-identical."""
    G, f, d = 2, 128, 128
    desc = P.make_desc(T=8, d_model=d, d_ff=f, n_experts=2, top_k=1, dtype="bf16")
    W = [torch.randn(G, f, d, device="cuda").bfloat16() for _ in range(2)] + [torch.randn(G, d, f, device="cuda").bfloat16()]
    before = [x.clone() for x in W]
    Z = [torch.zeros_like(x) for x in W]
    n = sum(x.numel() for x in W)
    Mo, Ve = torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    P.moe_expert_update(desc, P.make_opt(kind="adamw", lr=1e-2, weight_decay=0.0, step=5), *W, *Z, None, Mo, Ve)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(W, before))
    assert not Mo.any() and not Ve.any()


def test_update_E16_f2816_d1024_sampled():
    """16 experts, f=2816, d=1024 (the benchmark's shapes), bf16 with master, AdamW: a sample of
    200k parameters against the oracle."""
    G, f, d = 16, 2816, 1024
    torch.manual_seed(0)
    shapes = [(G, f, d), (G, f, d), (G, d, f)]
    mst = [torch.randn(s, device="cuda") * 0.05 for s in shapes]
    W = [x.bfloat16() for x in mst]
    Gd = [(torch.randn(s, device="cuda") * 0.01).bfloat16() for s in shapes]
    master = torch.cat([x.reshape(-1) for x in mst])
    n = master.numel()
    Mo = torch.randn(n, device="cuda") * 1e-3
    Ve = torch.rand(n, device="cuda") * 1e-4
    idx = torch.from_numpy(np.random.default_rng(5).choice(n, 200_000, replace=False)).cuda()
    g_flat = torch.cat([x.reshape(-1) for x in Gd]).float()
    src, m0, v0, g0 = (t[idx].double().cpu().numpy() for t in (master, Mo, Ve, g_flat))
    desc = P.make_desc(T=4096, d_model=d, d_ff=f, n_experts=G, top_k=2, dtype="bf16")
    log("update E=16 f=2816 d=1024 sampled")
    P.moe_expert_update(desc, P.make_opt(kind="adamw", lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1,
                                         step=4), *W, *Gd, master, Mo, Ve)
    torch.cuda.synchronize()
    p, m, v = U.adamw_step(src, g0, m0, v0, 1e-3, 0.9, 0.95, 1e-8, 0.1, 4)
    for name, got_t, want in (("master", master, p), ("m", Mo, m), ("v", Ve, v)):
        assert_close(name, got_t[idx].double().cpu().numpy(), want, TOL["f32"])
    assert_close("master step", master[idx].double().cpu().numpy() - src, p - src, STEP_TOL)
    w_flat = torch.cat([x.reshape(-1) for x in W]).float()[idx].cpu().numpy()
    ulp = bf16_ulp_diff(w_flat, round_to_bf16(p.astype(np.float32)))
    assert ulp.max() <= 1 and (ulp == 0).mean() > 0.99
