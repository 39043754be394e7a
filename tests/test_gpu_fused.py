"""GPU tests of the down projection fused with the fixed-order combine
(moe_fp4_grouped_gemm_combine), through the C ABI.

The fused kernel forms the same fp32 products in the same order as the
two-kernel path and sums each token's slots with the combine's fmaf chain,
so its output must equal moe_fp4_grouped_gemm + moe_combine_fixed_order bit
for bit; it is also checked against the fp64 oracle (row-relative 1e-2, as
the layer tests) and for bit-identical repeats."""
import numpy as np
import pytest
import torch

import synth
from tests import gpu_common as gc
from tests.gpu_common import log
from tests.test_gpu_layer import check_against_oracle, run_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def m():
    from paper_2609_15627_amd import moe
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return moe


def both_paths(m, cfg, inp, fmt="e4m3", weights=None):
    w = weights if weights is not None else gc.dev_expert_weights(inp.weights)
    x = gc.to_dev_bf16(inp.x)
    assert m.moe_fp4_grouped_gemm_combine_supported(cfg.T, cfg.H, cfg.I, cfg.NE, cfg.k_total, fmt)
    lf, of = run_layer(m, cfg, x, w, logits=inp.logits, fmt=fmt, fused=True)
    assert lf.fused and lf.partials is None
    lu, ou = run_layer(m, cfg, x, w, logits=inp.logits, fmt=fmt, fused=False)
    assert m.moe_last_variant() == m.VARIANT_STREAM
    return lf, of, lu, ou


@pytest.mark.parametrize("fmt", ["e4m3", "e2m1"])
@pytest.mark.parametrize("shape", [
    (37, 512, 384, 16, 4, 1),     # ragged tiles; K/32 = 12: steps of 128, odd step count
    (64, 1024, 256, 64, 8, 1),    # decode-like spread; K/32 = 8: steps of 128, even count
    (3, 256, 128, 8, 8, 1),       # k = E
    (1, 128, 128, 1, 1, 0),       # smallest shape: 8 workgroups, one row
    (50, 512, 1024, 32, 6, 1),    # K/32 = 32: steps of 256; top-6 + shared
    (17, 2048, 512, 128, 8, 0),   # many experts with one row, some empty
])
def test_fused_matches_unfused_and_oracle(m, shape, fmt):
    T, H, I, E, k, S = shape
    cfg = synth.LayerConfig("fused", T, H, E, k, I, S, "normal", sum(shape) + 1)
    inp = synth.make_inputs(cfg)
    log(f"fused {shape} {fmt}")
    lf, of, lu, ou = both_paths(m, cfg, inp, fmt)
    assert np.array_equal(gc.bf16_bits(of), gc.bf16_bits(ou)), "fused output differs from unfused"
    assert np.array_equal(lf.ids.cpu().numpy(), lu.ids.cpu().numpy())
    check_against_oracle(cfg, inp, lf, of, np.arange(cfg.T), fmt)


def test_fused_row_limit(m):
    """The largest batch whose rows fit the workgroup's LDS, I = 2048: every
    row's result for 16 columns per K half (2 x 64 bytes a row) plus two
    slots of scale rows for each of 16 waves (64 KiB), within 160 KiB."""
    cfg = synth.LayerConfig("fused_max", 85, 512, 256, 8, 2048, 1, "normal", 11)
    assert cfg.A == 765
    inp = synth.make_inputs(cfg)
    log(f"fused row limit A={cfg.A}")
    lf, of, lu, ou = both_paths(m, cfg, inp)
    assert np.array_equal(gc.bf16_bits(of), gc.bf16_bits(ou))
    check_against_oracle(cfg, inp, lf, of, np.arange(0, cfg.T, 7))
    assert not m.moe_fp4_grouped_gemm_combine_supported(86, 512, 2048, 257, 9, "e4m3")


def test_fused_decode_full_size(m):
    """The decode workload (T=64, H=4096, 256+1 experts, top-8, I=2048), as the
    benchmark runs it: bit-identical to the unfused path, to the oracle on
    sampled tokens, and over ten repeats."""
    cfg = synth.CONFIGS["decode"]
    inp = synth.make_inputs(cfg, lazy=True)
    weights = gc.dev_weights(cfg)
    log("fused decode: both paths")
    lf, of, lu, ou = both_paths(m, cfg, inp, weights=weights)
    first = gc.bf16_bits(of).copy()
    assert np.array_equal(first, gc.bf16_bits(ou))
    check_against_oracle(cfg, inp, lf, of, np.array([0, 21, 63]), named=True)
    x = gc.to_dev_bf16(inp.x)
    lg = torch.from_numpy(inp.logits).cuda()
    for _ in range(9):
        o2 = lf.forward(x, weights, logits=lg)
        torch.cuda.synchronize()
        assert np.array_equal(gc.bf16_bits(o2), first)
    log("fused decode: 10 runs bit-identical")


def test_fused_stages_and_graph(m):
    """Stage bits called one by one give the whole call's bits; so does a
    captured graph of the fused layer, replayed several times."""
    cfg = synth.LayerConfig("fused_st", 48, 1024, 64, 8, 512, 1, "normal", 5)
    inp = synth.make_inputs(cfg)
    w = gc.dev_expert_weights(inp.weights)
    x = gc.to_dev_bf16(inp.x)
    lg = torch.from_numpy(inp.logits).cuda()
    log("fused stages")
    layer = m.MoELayer(cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.n_shared, fused=True)
    ref = gc.bf16_bits(layer.forward(x, w, logits=lg)).copy()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(7)]
    out = layer.forward(x, w, logits=lg, events=ev)
    torch.cuda.synchronize()
    assert np.array_equal(gc.bf16_bits(out), ref)
    log("fused graph")
    layer.capture(x, w, logits=lg)
    for _ in range(3):
        layer.out.zero_()
        torch.cuda.synchronize()
        layer.replay()
        torch.cuda.synchronize()
        assert np.array_equal(gc.bf16_bits(layer.out), ref)


def test_fused_rejects(m):
    """Dims the fused kernel does not take: the tiled geometry (many rows per
    expert) and batches past the LDS limit; both report MOE_ERR_UNSUPPORTED."""
    assert not m.moe_fp4_grouped_gemm_combine_supported(600, 512, 1024, 2, 1, "e4m3")
    assert not m.moe_fp4_grouped_gemm_combine_supported(4096, 4096, 256, 256, 8, "e4m3")
    with pytest.raises(m.MoeError) as ei:
        m.MoELayer(600, 512, 2, 1, 1024, 0, fused=True)
    assert ei.value.status == m.MOE_ERR_UNSUPPORTED
    cfg = synth.LayerConfig("rej", 600, 512, 2, 1, 1024, 0, "normal", 3)
    inp = synth.make_inputs(cfg)
    x = gc.to_dev_bf16(inp.x)
    w = gc.dev_expert_weights(inp.weights)
    ids = torch.from_numpy(np.argmax(inp.logits, 1).astype(np.int32)[:, None]).cuda()
    tw = torch.ones((cfg.T, 1), dtype=torch.float32, device="cuda")
    _, offsets, srt, _ = m.moe_permute(ids, cfg.NE)
    with pytest.raises(m.MoeError) as ei:
        m.moe_fp4_grouped_gemm_combine(x, offsets, srt, *w, tw)
    assert ei.value.status == m.MOE_ERR_UNSUPPORTED
