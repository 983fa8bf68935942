"""The allocation-free dispatch (moe_permute_noalloc, for callers that cannot allocate device memory) against
moe_permute through the C ABI: bit-identical counts, offsets, both slot maps and gathered rows, on two calls in a
row on the same GPU, the second with a smaller input (its scratch keeps the first call's contents)."""
import numpy as np
import pytest
import torch

from paper_2506_02965_amd import pcmoe as P
from paper_2506_02965_amd.layer import MoELayer, upload
from paper_2506_02965_amd.synth import LayerConfig, make_inputs
from gpu_util import log

pytestmark = pytest.mark.gpu


def dispatch_both(cfg):
    inp = make_inputs(cfg, with_dy=False)
    w = upload(inp)
    layer = MoELayer(cfg, backward=False)
    layer.route(w)
    layer.permute(w)                      # moe_permute with its workspace
    T, k, d, lc = cfg.T, cfg.k, cfg.d, cfg.n_local
    dev = dict(device="cuda", dtype=torch.int32)
    counts, offsets = torch.full((lc,), -7, **dev), torch.full((lc + 1,), -7, **dev)
    r2s, s2r = torch.full((T * k,), -7, **dev), torch.full((T * k,), -7, **dev)
    xp = torch.zeros(T * k, d, device="cuda", dtype=layer.x_perm.dtype)
    P.moe_permute_noalloc(layer.desc, layer.topk_idx, w.x, counts, offsets, r2s, s2r, xp)
    torch.cuda.synchronize()
    n = int(layer.offsets[-1].item())
    assert torch.equal(counts, layer.counts[:lc]) and torch.equal(offsets, layer.offsets)
    assert torch.equal(r2s, layer.row_to_slot) and torch.equal(s2r, layer.slot_to_row)
    assert torch.equal(xp[:n], layer.x_perm[:n])
    return n


def test_permute_noalloc_matches_permute():
    big = LayerConfig("na1", T=8192, d=512, f=128, E=64, k=6, bias="zipf", seed=51)     # 48 blocks x 64 experts
    small = LayerConfig("na2", T=300, d=256, f=128, E=8, k=2, local_begin=2, local_count=4, seed=52)
    for cfg in (big, small):
        log(f"[noalloc] T={cfg.T} E={cfg.E} k={cfg.k} hosted={cfg.n_local}")
        n = dispatch_both(cfg)
        log(f"[noalloc] {n} hosted rows identical")
