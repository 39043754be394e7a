"""Pins of the oracle's BF16 contract (fmt='bf16', CPU only): x enters the
projections unquantised and the intermediate h is rounded once to bf16
before the down projection (the paper's accepted large-prefill arithmetic:
Large-M CK and the meaning of the earlier 6.42k result; Historical
down-consumer pilot, which consumes the already-rounded BF16 intermediate).

Hand-computed closed forms tell this mode apart from the MXFP8 contract and
from the unquantised reading; the explicit-loop brute force
(test_oracle_layer.py) covers it on random tiny layers."""
import numpy as np
import torch

import synth
from oracle import moe, mx


def _const_expert(h, i, code=2, scale=127):
    byte = code | (code << 4)
    return (np.full((1, 2 * i, h // 2), byte, np.uint8), np.full((1, 2 * i, h // 32), scale, np.uint8),
            np.full((1, h, i // 2), byte, np.uint8), np.full((1, h, i // 32), scale, np.uint8))


def test_h1_bf16_rounds_the_intermediate():
    """x = 0.5, every weight 1.0, H = I = 32: G = U = 16, h = 256 / (1 + e^-16)
    = 255.99997..., which bf16 rounds to 256 (spacing 1 in [128, 256)); so
    each partial is 32 * 256 = 8192 exactly, where the unquantised reading
    gives 8191.99908..."""
    x = np.full((1, 32), 0x3F00, np.uint16)
    w = _const_expert(32, 32)
    lg = np.zeros((1, 1), np.float32)
    r = moe.layer(x, *w, k=1, logits=lg, fmt="bf16", keep=True)
    e = r["per_expert"][0]
    assert np.all(e["g"] == 16.0) and np.all(e["u"] == 16.0)
    assert np.all(e["hd"] == 256.0)
    assert np.all(e["p"] == 8192.0)
    rx = moe.layer(x, *w, k=1, logits=lg, fmt=None, keep=True)
    assert np.all(np.abs(rx["per_expert"][0]["p"] - 8191.99908) < 1e-5)


def test_x_is_not_quantised():
    """x = bf16 0.30078125 (0x3E9A): the BF16 contract keeps it, so G = 32 * x =
    9.625 exactly; MXFP8 would quantise it to 0.3125 (block exponent -10,
    308 -> code 320), giving G = 10."""
    x = np.full((1, 32), 0x3E9A, np.uint16)
    assert mx.bf16_to_f64(x)[0, 0] == 0.30078125
    w = _const_expert(32, 32)
    lg = np.zeros((1, 1), np.float32)
    rb = moe.layer(x, *w, k=1, logits=lg, fmt="bf16", keep=True)
    assert np.all(rb["per_expert"][0]["g"] == 9.625)
    rq = moe.layer(x, *w, k=1, logits=lg, fmt="e4m3", keep=True)
    assert np.all(rq["per_expert"][0]["g"] == 10.0)


def test_h_rounding_matches_torch_bf16_cast():
    """The rounded intermediate equals torch's bf16 cast of h (which rounds
    through fp32) except where the fp32 value sits exactly on a bf16 midpoint
    (low 16 bits 0x8000: there the two roundings may differ); and everywhere
    it lies within half a bf16 spacing of h."""
    cfg = synth.LayerConfig("b16", 6, 64, 4, 2, 64, 1, "normal", 21)
    inp = synth.make_inputs(cfg)
    r = moe.layer(inp.x, *inp.weights, k=2, n_shared=1, logits=inp.logits, fmt="bf16", keep=True)
    checked = 0
    for e in r["per_expert"].values():
        h = e["h"]
        h32 = h.astype(np.float32)
        mid = (h32.view(np.uint32) & 0xFFFF) == 0x8000
        t = torch.from_numpy(h32).to(torch.bfloat16).to(torch.float64).numpy()
        assert np.array_equal(e["hd"][~mid], t[~mid])
        _, ex = np.frexp(h)
        assert np.all(np.abs(e["hd"] - h) <= np.ldexp(1.0, ex - 9))
        checked += int((~mid).sum())
    assert checked > 1000


def test_bound_against_unquantised_reading():
    """The only difference from the unquantised reading is the rounding of h
    (at most half a spacing, 2^-8 relative, per element: bf16 keeps 8
    significant bits), so each partial differs by at most
    2^-8 * sum_i |h_i| |W2_ni| (plus fp64 rounding)."""
    cfg = synth.LayerConfig("b16b", 5, 64, 4, 2, 96, 1, "normal", 22)
    inp = synth.make_inputs(cfg)
    rb = moe.layer(inp.x, *inp.weights, k=2, n_shared=1, logits=inp.logits, fmt="bf16", keep=True)
    rx = moe.layer(inp.x, *inp.weights, k=2, n_shared=1, logits=inp.logits, fmt=None, keep=True)
    w2all = [mx.dequant_fp4(inp.weights[2][e], inp.weights[3][e]) for e in range(cfg.NE)]
    for ex, e in rb["per_expert"].items():
        bound = np.abs(rx["per_expert"][ex]["h"]) @ np.abs(w2all[ex]).T * 2.0 ** -8
        d = np.abs(e["p"] - rx["per_expert"][ex]["p"])
        assert np.all(d <= bound * (1 + 1e-9) + 1e-9)
    assert not np.array_equal(rb["out_f64"], rx["out_f64"])


def test_metamorphic_scale_bumps_double_output_bf16():
    """W2 scales + 1 and up-row scales + 1 each double every output exactly
    (doubling commutes with the bf16 rounding of h)."""
    cfg = synth.LayerConfig("b16m", 6, 64, 4, 2, 64, 1, "normal", 23)
    inp = synth.make_inputs(cfg)
    w13, w13s, w2, w2s = inp.weights
    kw = dict(k=2, n_shared=1, logits=inp.logits, fmt="bf16")
    base = moe.layer(inp.x, w13, w13s, w2, w2s, **kw)
    assert np.array_equal(moe.layer(inp.x, w13, w13s, w2, w2s + 1, **kw)["out_f64"],
                          2 * base["out_f64"])
    up = w13s.copy()
    up[:, 64:] += 1
    assert np.array_equal(moe.layer(inp.x, w13, up, w2, w2s, **kw)["out_f64"], 2 * base["out_f64"])
