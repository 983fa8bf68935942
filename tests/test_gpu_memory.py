"""One party's expert-layer training step on the GPU: the peak device memory torch reports agrees with the
footprint accounted from the library's own buffer and workspace sizes, for all experts hosted and for a shard."""
import dataclasses

import pytest
import torch

from paper_2506_02965_amd import pcmoe as P
from paper_2506_02965_amd.layer import MoELayer, upload, training_footprint
from paper_2506_02965_amd.synth import LayerConfig, make_inputs
from gpu_util import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("local", [16, 4])
def test_peak_memory_matches_accounting(local):
    cfg = LayerConfig("mem", T=2048, d=512, f=512, E=16, k=2, local_count=local, seed=31)
    log(f"memory local={local}")
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    start = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    inp = make_inputs(cfg, with_dy=True)
    w = upload(inp)
    layer = MoELayer(cfg, backward=True, router_backward=True)
    layer.init_update_state(w, master=True)
    layer.dlogits.zero_()
    layer.forward(w)
    layer.combine_bwd(w.dy)
    layer.ffn_bwd(w, w.dy)
    if local == cfg.E:
        layer.route_bwd(w)
    layer.permute_bwd(w)
    layer.update(w, P.make_opt(kind="adamw", lr=1e-4, step=1))
    torch.cuda.synchronize()
    peak = torch.cuda.max_memory_allocated() - start
    acc = training_footprint(cfg, local)["total"]
    # the caching allocator rounds every block up to 512 bytes
    assert acc <= peak <= acc * 1.02 + 64 * 1024, (peak, acc)
