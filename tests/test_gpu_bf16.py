"""GPU parity of the BF16 contract (MOE_ACT_BF16) against the fp64 oracle in
the same mode (x unquantised, FP4 weights exact, h rounded once to bf16),
through the C ABI.

Bar, from the arithmetic: the output is rounded to bf16 (8 significant
bits: at most 2^-8 of a row's largest value); h can land one bf16 step away
from the oracle's where the GPU's fp32 value and the oracle's fp64 value
straddle a rounding midpoint (2^-8 of one element, about 2^-8 /
sqrt(I * k_total) of a row, measured below 1e-3 on the partials); fp32
accumulation adds about 1e-6. So row-relative error <= 2^-8 + 1e-3 (5e-3),
h bits equal except rare flips of one step plus 1e-5 of the
row's largest |h| (fp32 accumulation where G nearly cancels; values below
1e-30, where the GPU's fp32 SwiGLU underflows to zero, aside), partials within
1e-3 row-relative; routing and permutation bit-exact; repeats bit-identical.
Also the quality comparison the contract exists for: against the unquantised
reading (no rounding of x or h), the BF16 contract's error is a fraction of
the MXFP8 contract's."""
import numpy as np
import pytest
import torch

import synth
from oracle import moe as omoe
from oracle import mx
from tests import gpu_common as gc
from tests.gpu_common import log

pytestmark = pytest.mark.gpu

TOL = 5e-3


@pytest.fixture(scope="module")
def m():
    from paper_2609_15627_amd import moe
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return moe


def run(m, cfg, inp, weights=None, fmt="bf16"):
    w = weights if weights is not None else gc.dev_expert_weights(inp.weights)
    layer = m.MoELayer(cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.n_shared, fmt)
    out = layer.forward(gc.to_dev_bf16(inp.x), w, logits=torch.from_numpy(inp.logits).cuda())
    torch.cuda.synchronize()
    return layer, out


def check(cfg, inp, layer, out, tokens):
    ref = omoe.layer(inp.x, *inp.weights, k=cfg.k, n_shared=cfg.n_shared, logits=inp.logits,
                     fmt="bf16", tokens=tokens, keep=True)
    y = gc.bf16_to_f64(gc.bf16_bits(out)[tokens])
    err = gc.rowrel(y, ref["out_f64"])
    P = layer.partials.view(cfg.T, cfg.k_total, cfg.H).cpu().numpy()[tokens]
    perr = gc.rowrel(P.reshape(-1, cfg.H), ref["p_slots"].reshape(-1, cfg.H))
    flips = total = nbad = 0
    worst = 0.0
    badmsg = ""
    if len(tokens) == cfg.T:
        hq = layer.workspace_view(2)[: cfg.A * cfg.I * 2].cpu().numpy().view(np.uint16)
        hq = hq.reshape(cfg.A, cfg.I)
        for r in ref["per_expert"].values():
            g, o = hq[r["rows"]], r["hq"]
            gv, ov = mx.bf16_to_f64(g), mx.bf16_to_f64(o)
            big = np.maximum(np.abs(gv), np.abs(ov))
            _, ex = np.frexp(big)
            # one bf16 step, plus fp32 accumulation error of G and U, which is
            # relative to the row's largest products (where G nearly cancels,
            # h can move several steps); values below 1e-30 are where the GPU's
            # fp32 SwiGLU underflows to zero for G < -88
            rowmax = np.abs(r["h"]).max(axis=1, keepdims=True)
            excess = np.abs(gv - ov) - np.ldexp(1.0, ex - 8)
            worst = max(worst, float((excess / np.maximum(rowmax, 1e-300)).max()))
            bad = (excess > 1e-5 * rowmax) & (big > 1e-30)
            nbad += int(bad.sum())
            if bad.any() and not badmsg:
                badmsg = f"h: {gv[bad][:6]} vs {ov[bad][:6]} (row max {rowmax.max():.3g})"
            flips += int(((g != o) & (big > 1e-30)).sum())
            total += g.size
    log(f"  rowrel={err:.3e} (bar {TOL:g}) partials {perr:.2e}; h flips {flips}/{total}, "
        f"largest h excess over one step {worst:.1e} of the row max; {nbad} beyond the bound")
    assert nbad == 0, badmsg
    assert flips <= 1e-3 * max(total, 1), (flips, total)
    assert err <= TOL
    assert perr <= 1e-3
    return ref, err


@pytest.mark.parametrize("shape", [
    (37, 512, 384, 16, 4, 1),     # ragged: ~10 rows per expert, 6 h tiles
    (200, 384, 384, 4, 2, 0),     # two row tiles per expert, ragged tail
    (64, 1024, 256, 64, 8, 1),    # decode-like spread
    (3, 256, 128, 8, 8, 1),       # k = E
    (1, 128, 128, 1, 1, 0),       # smallest shape: 4 K steps (fewer than the ring)
    (300, 1024, 512, 4, 2, 1),    # ~150-300 rows per expert
    (130, 512, 512, 2, 1, 0),     # 128-row tile plus a 2-row tile
    (20, 384, 640, 8, 2, 0),      # streaming geometry, odd step counts (3 and 5 K steps)
])
def test_bf16_small_layers(m, shape):
    T, H, I, E, k, S = shape
    cfg = synth.LayerConfig("bf16", T, H, E, k, I, S, "normal", sum(shape) + 2)
    inp = synth.make_inputs(cfg)
    log(f"bf16 layer {shape}")
    layer, out = run(m, cfg, inp)
    # tiled from 64 rows per expert on average, else weight streaming
    tiled = cfg.T * cfg.k_total >= 64 * cfg.NE
    assert m.moe_last_variant() == (m.VARIANT_BF16 if tiled else m.VARIANT_BF16_STREAM)
    ref, _ = check(cfg, inp, layer, out, np.arange(cfg.T))
    assert np.array_equal(layer.ids.cpu().numpy(), ref["ids"])
    assert np.array_equal(layer.perm[2].cpu().numpy(), ref["sorted"])
    first = gc.bf16_bits(out).copy()
    w = gc.dev_expert_weights(inp.weights)
    for _ in range(3):
        o2 = layer.forward(gc.to_dev_bf16(inp.x), w, logits=torch.from_numpy(inp.logits).cuda())
        torch.cuda.synchronize()
        assert np.array_equal(gc.bf16_bits(o2), first), "repeat differs"


def test_bf16_quality_against_unquantised(m):
    """Error against the unquantised reading (Oracle-X, reported, not the
    parity reference): the BF16 contract's (output and h rounding, each up to
    2^-8) stays within 1e-2 and is at most a quarter of the MXFP8
    contract's on the same layer."""
    cfg = synth.LayerConfig("bf16q", 48, 1024, 16, 4, 512, 1, "normal", 31)
    inp = synth.make_inputs(cfg)
    refx = omoe.layer(inp.x, *inp.weights, k=cfg.k, n_shared=cfg.n_shared, logits=inp.logits,
                      fmt=None)
    errs = {}
    for fmt in ("bf16", "e4m3"):
        log(f"quality {fmt}")
        _, out = run(m, cfg, inp, fmt=fmt)
        errs[fmt] = gc.rowrel(gc.bf16_to_f64(gc.bf16_bits(out)), refx["out_f64"])
    log(f"  vs unquantised: bf16 {errs['bf16']:.2e}, mxfp8 {errs['e4m3']:.2e}")
    assert errs["bf16"] <= 1e-2
    assert errs["bf16"] * 4 <= errs["e4m3"]


@pytest.mark.parametrize("name,ntok", [("decode", 3), ("prefill8k", 2)])
def test_bf16_full_size(m, name, ntok):
    """Full-size workloads under the BF16 contract: sampled tokens against the
    oracle, three runs bit-identical."""
    cfg = synth.CONFIGS[name]
    inp = synth.make_inputs(cfg, lazy=True)
    weights = gc.dev_weights(cfg)
    log(f"bf16 full {name}")
    layer, out = run(m, cfg, inp, weights=weights)
    ids = layer.ids.cpu().numpy()
    rng = np.random.default_rng(5)
    tokens = np.unique(np.concatenate([[0, cfg.T - 1], rng.choice(cfg.T, ntok, replace=False)]))
    check(cfg, inp, layer, out, tokens)
    first = gc.bf16_bits(out).copy()
    x = gc.to_dev_bf16(inp.x)
    lg = torch.from_numpy(inp.logits).cuda()
    for _ in range(2):
        o2 = layer.forward(x, weights, logits=lg)
        torch.cuda.synchronize()
        assert np.array_equal(gc.bf16_bits(o2), first)
    assert ids.shape == (cfg.T, cfg.k_total)


def test_bf16_streaming_skewed(m):
    """Zipf-skewed routing through the BF16 streaming geometry: empty
    experts, experts of one row and experts of several 16-row tiles."""
    cfg = synth.LayerConfig("bf16skew", 48, 512, 32, 4, 384, 1, "zipf", 9, zipf_empty=6)
    inp = synth.make_inputs(cfg)
    log("bf16 streaming skewed")
    layer, out = run(m, cfg, inp)
    assert m.moe_last_variant() == m.VARIANT_BF16_STREAM
    ref, _ = check(cfg, inp, layer, out, np.arange(cfg.T))
    counts = np.bincount(ref["ids"].ravel(), minlength=cfg.NE)
    assert (counts == 0).any() and counts.max() > 16, counts
    first = gc.bf16_bits(out).copy()
    o2 = layer.forward(gc.to_dev_bf16(inp.x), gc.dev_expert_weights(inp.weights),
                       logits=torch.from_numpy(inp.logits).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(gc.bf16_bits(o2), first)
