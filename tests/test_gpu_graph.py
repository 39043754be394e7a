"""HIP-graph capture of the whole layer (one graph launch per step).

A captured forward must give the same bits as the eager forward on every
replay, with eager work and synchronisations between the replays (graph
replays have been seen to differ from the first when a graph holds memset
nodes; the layer's kernels clear what they need themselves). Covers both
GEMM geometries (the persistent tiled kernels leave their work queue at zero
at the end of every launch, which replays rely on), new inputs copied into
the captured tensors, and parity with the oracle for the replayed output."""
import numpy as np
import pytest
import torch

import synth
from oracle import moe as omoe
from tests import gpu_common as gc
from tests.gpu_common import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def m():
    from paper_2609_15627_amd import moe
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return moe


@pytest.mark.parametrize("shape,variant", [
    ((64, 1024, 256, 64, 8, 1), 1),    # decode-like: weight-streaming geometry
    ((600, 512, 1024, 2, 1, 0), 2),    # tiled geometry, persistent kernels
])
def test_graph_replays_match_eager(m, shape, variant):
    T, H, I, E, k, S = shape
    cfg = synth.LayerConfig("small", T, H, E, k, I, S, "normal", 11)
    inp = synth.make_inputs(cfg)
    log(f"graph: shape={shape}")
    x = gc.to_dev_bf16(inp.x)
    w = gc.dev_expert_weights(inp.weights)
    lg = torch.from_numpy(inp.logits).cuda()
    eager = m.MoELayer(T, H, E, k, I, S, "e4m3")
    ref = eager.forward(x, w, logits=lg).clone()
    torch.cuda.synchronize()
    assert m.moe_last_variant() == variant

    layer = m.MoELayer(T, H, E, k, I, S, "e4m3")
    out = layer.capture(x, w, logits=lg)
    for r in range(4):
        out = layer.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {r} differs from the eager forward"
        eager.forward(x, w, logits=lg)  # eager work between replays
        torch.cuda.synchronize()

    # new inputs through the captured tensors
    cfg2 = synth.LayerConfig("small", T, H, E, k, I, S, "normal", 12)
    inp2 = synth.make_inputs(cfg2)
    x.copy_(gc.to_dev_bf16(inp2.x))
    lg.copy_(torch.from_numpy(inp2.logits).cuda())
    out = layer.replay()
    torch.cuda.synchronize()
    ref2 = eager.forward(x, w, logits=lg)
    torch.cuda.synchronize()
    assert torch.equal(out, ref2)
    tokens = list(range(min(T, 8)))
    o = omoe.layer(inp2.x, *inp.weights, k=k, n_shared=S, logits=inp2.logits, fmt="e4m3",
                   tokens=tokens)
    err = gc.rowrel(gc.bf16_to_f64(gc.bf16_bits(out)[tokens]), o["out_f64"])
    log(f"  replay with new inputs: rowrel={err:.3e}")
    assert err <= 1e-2
