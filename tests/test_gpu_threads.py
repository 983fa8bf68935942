"""Reentrancy of the C ABI: two host threads drive two different layers at the same time, each on its own
stream, and every output matches a run of that layer alone bit for bit. The library's only process-wide
state is set up once (kernel attributes, tuning switches, device properties) and every call enqueues its
work on the caller's stream."""
import threading

import pytest
import torch

from paper_2506_02965_amd.layer import MoELayer, upload
from paper_2506_02965_amd.synth import LayerConfig, make_inputs
from gpu_util import log

pytestmark = pytest.mark.gpu

OUTPUTS = ("logits", "topk_idx", "topk_w", "row_to_slot", "slot_to_row", "y", "dgate", "dw_gate", "dw_up", "dw_down",
           "dw_router", "dx")


def test_two_threads_two_streams():
    cfgs = [LayerConfig("th0", T=1000, d=256, f=384, E=16, k=2, n_shared=1, seed=31),
            LayerConfig("th1", T=700, d=512, f=256, E=8, k=3, seed=32)]
    weights = [upload(make_inputs(c, with_dy=True)) for c in cfgs]
    ref = []
    for c, w in zip(cfgs, weights):
        layer = MoELayer(c)
        layer.forward(w)
        layer.backward(w)
        torch.cuda.synchronize()
        ref.append({n: getattr(layer, n).clone() for n in OUTPUTS})
        del layer
    layers = [MoELayer(c) for c in cfgs]
    streams = [torch.cuda.Stream() for _ in cfgs]  # default priority
    torch.cuda.synchronize()
    errors = []

    def work(i):
        try:
            with torch.cuda.stream(streams[i]):
                for _ in range(4):
                    layers[i].forward(weights[i])
                    layers[i].backward(weights[i])
            streams[i].synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    log("[threads] two layers on two streams from two host threads")
    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(cfgs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    for i, layer in enumerate(layers):
        for n in OUTPUTS:
            assert torch.equal(getattr(layer, n), ref[i][n]), f"layer {i}: {n} differs from its single-thread run"
