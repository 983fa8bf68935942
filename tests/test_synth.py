"""The seeded input generator: determinism, storage rounding and the workload recipes."""
import numpy as np
import torch

from paper_2506_02965_amd.synth import CONFIGS, LayerConfig, make_inputs, round_to_bf16, zipf_logit_bias, bf16_bits


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    # include exact halfway cases (ties to even)
    half = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8)], np.float32)
    a = np.concatenate([a, half])
    ref = torch.from_numpy(a).to(torch.bfloat16).float().numpy()
    assert np.array_equal(round_to_bf16(a), ref)
    assert np.array_equal(bf16_bits(ref), torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))


def test_deterministic_and_keyed():
    cfg = LayerConfig("t", T=64, d=128, f=128, E=4, k=2, n_shared=1, seed=3)
    a, b = make_inputs(cfg), make_inputs(cfg)
    for n in ("x", "dy", "w_router", "w_gate", "w_up", "w_down"):
        assert np.array_equal(getattr(a, n), getattr(b, n))
    # expert e's weights do not depend on how many experts are hosted (keyed by global id)
    shard = make_inputs(cfg.scaled(local_begin=2, local_count=2, n_shared=0))
    assert np.array_equal(shard.w_gate[0], a.w_gate[2])
    assert np.array_equal(round_to_bf16(a.x), a.x)


def test_variances():
    cfg = LayerConfig("v", T=2048, d=256, f=512, E=8, k=2, seed=1)
    inp = make_inputs(cfg)
    assert abs(inp.x.std() - 1) < 0.01
    assert abs(inp.w_gate.std() * np.sqrt(256) - 1) < 0.01
    assert abs(inp.w_down.std() * np.sqrt(512) - 1) < 0.01
    assert abs(inp.w_router.std() * np.sqrt(256) - 1) < 0.05


def test_zipf_bias():
    b = zipf_logit_bias(64)[0].astype(np.float64)
    H = sum(r ** -1.1 for r in range(1, 65))
    assert abs(H - 3.99205) < 1e-4
    assert abs(b[0] - (-np.log(H))) < 1e-6 and abs(b[63] - (-1.1 * np.log(64) - np.log(H))) < 1e-5
    assert np.all(np.diff(b) < 0)


def test_config_table():
    assert CONFIGS[1].dtype == "f32" and not CONFIGS[1].backward
    assert CONFIGS[3].n_local == 16 and CONFIGS[3].bias_groups == 4 and not CONFIGS[3].router_backward
    assert CONFIGS[5].n_groups == 66
    for c in CONFIGS.values():
        assert c.d % 128 == 0 and c.f % 128 == 0
