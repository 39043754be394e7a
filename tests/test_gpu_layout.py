"""Output-column fingerprints through the GPU path (the paper located its W2
row-order fault this way: Correctness recovery / W2 permutation).

With the column-fingerprint weights of tests/layout_fingerprint.py every fp32
partial is an exact value that names the W2 row it came from. On each GEMM
geometry and activation format, every partial row must decode to the
identity (no N-tile, 16-row block or column permutation) and equal the
oracle's partial exactly."""
import numpy as np
import pytest
import torch

import synth
from oracle import moe as omoe
from tests import gpu_common as gc
from tests import layout_fingerprint as fp
from tests.gpu_common import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def m():
    from paper_2609_15627_amd import moe
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return moe


@pytest.mark.parametrize("fmt", ["e4m3", "e2m3", "e2m1", "bf16"])
@pytest.mark.parametrize("T,H,I,variants", [
    (5, 256, 128, (1, 5)),       # weight-streaming geometry (MX / BF16 contract)
    (300, 512, 512, (2, 3)),     # LDS-tiled geometry: full row tiles and a ragged one
    (300, 1024, 256, (6, 3)),    # tiled stage 1, short-K stage 2 (I = 256)
    (300, 512, 384, (4, 3)),     # tiled stage 1, streaming stage 2 (I = 384)
    (300, 768, 128, (6, 3)),     # streaming stage 1 (H = 768), short-K stage 2 (I = 128)
])
def test_partials_decode_to_identity(m, T, H, I, variants, fmt):
    log(f"layout fingerprint T={T} H={H} I={I} {fmt}")
    w_np = fp.weights(H, I)
    w = gc.dev_expert_weights(w_np)
    x = gc.to_dev_bf16(fp.x_bits(T, H))
    layer = m.MoELayer(T, H, 1, 1, I, 0, fmt)
    layer.forward(x, w, logits=torch.zeros((T, 1), dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    assert m.moe_last_variant() == variants[1 if fmt == "bf16" else 0]
    P = layer.partials.cpu().numpy().astype(np.float64)
    ref = omoe.layer(fp.x_bits(2, H), *w_np, k=1, logits=np.zeros((2, 1), np.float32),
                     fmt=fmt, keep=True)["p_slots"][0, 0]
    assert fp.decode(ref, H).tolist() == list(range(H))
    for r in (0, T // 2, T - 1):
        got = fp.decode(P[r], H)
        bad = np.nonzero(got != np.arange(H))[0]
        assert bad.size == 0, f"row {r}: columns {bad[:8].tolist()} decode to {got[bad[:8]].tolist()}"
    assert np.array_equal(P, np.broadcast_to(ref, P.shape)), "partials differ from the exact value"
