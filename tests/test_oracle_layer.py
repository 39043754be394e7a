"""Pins of the oracle's layer (CPU only).

Hand-derived closed forms (tests/golden/hand_cases.json), brute force by
explicit loops (tests/bruteforce.py), special cases that reduce to textbook
routines (a dense SwiGLU MLP, the full softmax), invariants, and exact
metamorphic relations.
"""
import json
import os

import numpy as np
import pytest
import scipy.special

import synth
from oracle import moe, mx
from tests import bruteforce as bf
from tests.conftest import GOLDEN

HAND = json.load(open(os.path.join(GOLDEN, "hand_cases.json")))


def _const_expert(h, i, code=2, scale=127, w2_scale=None):
    byte = code | (code << 4)
    w13 = np.full((2 * i, h // 2), byte, np.uint8)
    w13s = np.full((2 * i, h // 32), scale, np.uint8)
    w2 = np.full((h, i // 2), byte, np.uint8)
    w2s = np.full((h, i // 32), scale if w2_scale is None else w2_scale, np.uint8)
    return w13, w13s, w2, w2s


def _stack(experts):
    return tuple(np.stack(a) for a in zip(*experts))


def test_h1_closed_form():
    c = HAND["H1"]
    x = np.full((1, 32), 0x3F00, np.uint16)          # bf16 0.5
    w = _stack([_const_expert(32, 32)])
    r = moe.layer(x, *w, k=1, logits=np.zeros((1, 1), np.float32), fmt="e4m3", keep=True)
    assert r["xs"].tolist() == [[c["x_scale_byte"]]]
    assert np.all(r["xq"] == c["x_code_e4m3"])
    assert np.all(r["per_expert"][0]["hs"] == c["h_scale_byte"])
    assert np.all(r["out_f64"] == c["out"])
    assert np.all(r["out"] == c["out_bf16_bits"])
    rx = moe.layer(x, *w, k=1, logits=np.zeros((1, 1), np.float32), fmt=None)
    assert np.allclose(rx["out_f64"], c["out_unquantised"], rtol=0, atol=1e-5)


def test_h1_distinguishes_floor_scale_rule():
    """The OCP floor rule (X = f - emax) would saturate h at 448 and give 7168."""
    h = 256.0 / (1.0 + np.exp(-16.0))
    codes, sb = mx.mx_quantize(np.full((1, 32), h), "e4m3")
    assert 32 * mx.mx_dequantize(codes, sb, "e4m3")[0, 0] == 8192.0
    assert 32 * 448 * 0.5 == 7168.0 and mx.mx_scale_exponent(h, "e4m3") == 0


def test_h2_tie_and_combine():
    c = HAND["H2"]
    x = np.full((1, 32), 0x3F00, np.uint16)
    e0 = _const_expert(32, 32)
    e2 = _const_expert(32, 32, w2_scale=128)
    w = _stack([e0, e0, e2, e0])
    logits = np.array([[1, 3, 3, 0]], np.float32)
    r = moe.layer(x, *w, k=2, logits=logits, fmt="e4m3")
    assert r["ids"].tolist() == [c["ids"]]
    assert r["w"].tolist() == [c["w"]]
    assert np.all(r["out_f64"] == c["out"])


def test_h4_router_projection_closed_form():
    """The router projection (the "Router" box of the layer figure) on the
    hand case H4: exact in fp64 where an fp32 sum would drop the 2^-30 term,
    and row 0 tells an [E, H] reading of the router matrix from an [H, E] one."""
    c = HAND["H4"]
    x = np.array(c["x_bits"], np.uint16)
    wr = np.repeat(np.array(c["wr_row_bits"], np.uint16)[:, None], x.shape[1], axis=1)
    lg = moe.router_logits(x, wr)
    assert lg.tolist() == c["logits"]
    # the 2^-30 term really is invisible to an fp32 sum
    assert np.float32(1.0) + np.float32(2.0 ** -30) == np.float32(1.0)
    # and the layer routes on these logits when given router weights
    w = _stack([_const_expert(64, 32)] * 3)
    r = moe.layer(x, *w, k=1, wr_bits=wr, fmt="e4m3")
    assert r["ids"].ravel().tolist() == [2, 2]
    assert r["logits_f64"].tolist() == c["logits"]


@pytest.mark.parametrize("shape", [(1, 8, 1), (3, 32, 5), (4, 64, 7), (2, 96, 16)])
def test_router_projection_brute_force(shape):
    """Explicit loops over the bf16 fields with exactly rounded sums, on random
    bf16 values spanning several binades (products of two bf16 values are exact
    in fp64, so the oracle is within a few ulps of the exact sum)."""
    t, h, e = shape
    rng = np.random.default_rng(sum(shape))
    xf = rng.standard_normal((t, h)).astype(np.float32) * np.float32(2.0) ** rng.integers(-8, 8, (t, h))
    wf = rng.standard_normal((e, h)).astype(np.float32) * np.float32(0.02)
    xb, wb = synth.f32_to_bf16_bits(xf), synth.f32_to_bf16_bits(wf)
    lg = moe.router_logits(xb, wb)
    ref = np.array(bf.router_logits(xb.tolist(), wb.tolist()))
    scale = np.abs(mx.bf16_to_f64(xb)) @ np.abs(mx.bf16_to_f64(wb)).T
    assert lg.shape == (t, e)
    assert np.all(np.abs(lg - ref) <= 4 * h * 2.0 ** -53 * scale)


def test_h3_permutation():
    c = HAND["H3"]
    counts, offsets, srt, pos = moe.permute(np.array(c["ids"]), 3)
    assert counts.tolist() == c["counts"] and offsets.tolist() == c["offsets"]
    assert srt.tolist() == c["sorted"] and pos.tolist() == c["pos"]


def test_route_ties_lower_id_and_order():
    lg = np.array([[0.5, 2.0, 2.0, -1.0, 2.0], [0, 0, 0, 0, 0]], np.float32)
    ids, w = moe.route_topk(lg, 3)
    assert ids.tolist() == [[1, 2, 4], [0, 1, 2]]
    assert np.allclose(w, 1 / 3, rtol=0, atol=1e-15)
    ids, w = moe.route_topk(lg, 2, n_shared=1)
    assert ids.tolist() == [[1, 2, 5], [0, 1, 5]] and w[:, 2].tolist() == [1.0, 1.0]


def test_route_k_equals_e_is_full_softmax():
    lg = np.random.default_rng(0).standard_normal((50, 16)).astype(np.float32)
    ids, w = moe.route_topk(lg, 16)
    sm = scipy.special.softmax(lg.astype(np.float64), axis=1)
    assert np.allclose(np.take_along_axis(sm, ids, 1), w, rtol=1e-13, atol=0)


def test_route_invariants_decode_shape():
    cfg = synth.CONFIGS["decode"]
    lg = synth.gen_logits(cfg)
    ids, w = moe.route_topk(lg, cfg.k, cfg.n_shared)
    assert np.allclose(w[:, :cfg.k].sum(1), 1.0, rtol=0, atol=1e-14)
    routed = ids[:, :cfg.k]
    assert all(len(set(r)) == cfg.k for r in routed.tolist())
    sel = np.take_along_axis(lg, routed, 1)
    assert np.all(np.diff(sel, axis=1) <= 0)
    # nothing left out beats the k-th pick
    masked = lg.copy()
    np.put_along_axis(masked, routed, -np.inf, 1)
    assert np.all(masked.max(1) <= sel[:, -1])
    # brute-force route on a few tokens
    for t in range(0, cfg.T, 9):
        order = sorted(range(cfg.E), key=lambda e: (-float(lg[t, e]), e))[:cfg.k]
        assert ids[t, :cfg.k].tolist() == order


def test_permute_brute_force_and_invariants():
    rng = np.random.default_rng(5)
    for t, k, ne in [(1, 1, 1), (7, 3, 5), (64, 9, 257), (300, 8, 17)]:
        ids = rng.integers(0, ne, (t, k))
        counts, offsets, srt, pos = moe.permute(ids, ne)
        flat = ids.reshape(-1)
        assert srt.tolist() == sorted(range(flat.size), key=lambda a: (flat[a], a))
        assert counts.sum() == flat.size and offsets[-1] == flat.size
        assert np.array_equal(srt[pos], np.arange(flat.size))
        assert np.array_equal(np.bincount(srt // k, minlength=t), np.full(t, k))


def _tiny_case(seed, t, h, i, e, k, n_shared):
    cfg = synth.LayerConfig("bf", t, h, e, k, i, n_shared, "normal", seed)
    inp = synth.make_inputs(cfg)
    return cfg, inp


@pytest.mark.parametrize("fmt", ["e4m3", "e2m3", "e2m1", "bf16", None])
@pytest.mark.parametrize("shape", [(3, 32, 32, 4, 2, 0), (2, 64, 32, 3, 1, 1), (4, 32, 64, 4, 4, 1)])
def test_brute_force_layer(fmt, shape):
    """Explicit-loop layer agrees with the numpy oracle to 1e-12 (relative to the row max)."""
    cfg, inp = _tiny_case(11, *shape)
    r = moe.layer(inp.x, *inp.weights, k=cfg.k, n_shared=cfg.n_shared, logits=inp.logits, fmt=fmt)
    x = mx.bf16_to_f64(inp.x).tolist()
    lg = inp.logits.astype(np.float64).tolist()
    w13, w13s, w2, w2s = (a.tolist() for a in inp.weights)
    ref = np.array(bf.layer(x, lg, w13, w13s, w2, w2s, cfg.k, cfg.n_shared, fmt))
    scale = np.abs(ref).max(axis=1, keepdims=True)
    assert np.all(np.abs(r["out_f64"] - ref) <= 1e-12 * scale)


def test_k1_single_expert_is_dense_swiglu_mlp():
    """E=1, k=1, no activation quantisation: the layer is silu(x W1^T) * (x W3^T) W2^T."""
    cfg = synth.LayerConfig("mlp", 5, 64, 1, 1, 96, 0, "normal", 3)
    inp = synth.make_inputs(cfg)
    r = moe.layer(inp.x, *inp.weights, k=1, logits=inp.logits, fmt=None)
    tab = np.array(bf.paper_e2m1_table())
    w13, w13s, w2, w2s = (a[0] for a in inp.weights)

    def deq(p, s):
        codes = np.stack([p & 15, p >> 4], -1).reshape(p.shape[0], -1)
        return tab[codes] * np.repeat(2.0 ** (s.astype(np.float64) - 127), 32, axis=1)

    W13, W2 = deq(w13, w13s), deq(w2, w2s)
    x = inp.x.astype(np.uint32) << 16
    x = x.view(np.float32).astype(np.float64)
    g, u = x @ W13[:96].T, x @ W13[96:].T
    want = (g * scipy.special.expit(g) * u) @ W2.T
    assert np.allclose(r["out_f64"], want, rtol=1e-12, atol=1e-9)


def test_metamorphic_scale_bumps_double_output():
    cfg = synth.LayerConfig("mm", 6, 64, 4, 2, 64, 1, "normal", 7)
    inp = synth.make_inputs(cfg)
    w13, w13s, w2, w2s = inp.weights
    base = moe.layer(inp.x, w13, w13s, w2, w2s, k=2, n_shared=1, logits=inp.logits)
    r2 = moe.layer(inp.x, w13, w13s, w2, w2s + 1, k=2, n_shared=1, logits=inp.logits)
    assert np.array_equal(r2["out_f64"], 2 * base["out_f64"])
    up_bump = w13s.copy()
    up_bump[:, 64:] += 1                    # up rows only: h doubles, codes unchanged
    r3 = moe.layer(inp.x, w13, up_bump, w2, w2s, k=2, n_shared=1, logits=inp.logits)
    assert np.array_equal(r3["out_f64"], 2 * base["out_f64"])
    gate_bump = w13s.copy()
    gate_bump[:, :64] += 1                  # gate rows: not a linear change
    r4 = moe.layer(inp.x, w13, gate_bump, w2, w2s, k=2, n_shared=1, logits=inp.logits)
    assert not np.array_equal(r4["out_f64"], 2 * base["out_f64"])


def test_metamorphic_token_and_expert_relabel():
    cfg = synth.LayerConfig("mm2", 9, 64, 5, 2, 32, 1, "normal", 8)
    inp = synth.make_inputs(cfg)
    base = moe.layer(inp.x, *inp.weights, k=2, n_shared=1, logits=inp.logits)
    perm = np.random.default_rng(0).permutation(cfg.T)
    r = moe.layer(inp.x[perm], *inp.weights, k=2, n_shared=1, logits=inp.logits[perm])
    assert np.array_equal(r["out_f64"], base["out_f64"][perm])
    # relabel routed experts (shared stays last)
    rel = np.random.default_rng(1).permutation(cfg.E)
    inv = np.argsort(rel)
    w = [np.concatenate([a[:cfg.E][inv], a[cfg.E:]]) for a in inp.weights]
    r = moe.layer(inp.x, *w, k=2, n_shared=1, logits=inp.logits[:, inv])
    assert np.allclose(r["out_f64"], base["out_f64"], rtol=1e-13, atol=0)


def test_token_subset_matches_full():
    cfg = synth.LayerConfig("sub", 12, 64, 6, 3, 32, 1, "normal", 9)
    inp = synth.make_inputs(cfg)
    full = moe.layer(inp.x, *inp.weights, k=3, n_shared=1, logits=inp.logits)
    toks = np.array([7, 0, 11])
    sub = moe.layer(inp.x, *inp.weights, k=3, n_shared=1, logits=inp.logits, tokens=toks)
    assert np.array_equal(sub["out"], full["out"][toks])


def test_lazy_weights_equal_stacked():
    cfg = synth.LayerConfig("lz", 4, 64, 3, 2, 32, 1, "normal", 2)
    stacked = synth.gen_all_experts(cfg)
    lazy = synth.lazy_weights(cfg)
    for e in range(cfg.NE):
        for a, b in zip(stacked, lazy):
            assert np.array_equal(a[e], b[e])


def test_quantised_close_to_unquantised():
    """MXFP8 activations change the layer by a few percent at most (sanity, not a pin)."""
    cfg = synth.LayerConfig("q", 8, 256, 4, 2, 128, 1, "normal", 4)
    inp = synth.make_inputs(cfg)
    q = moe.layer(inp.x, *inp.weights, k=2, n_shared=1, logits=inp.logits, fmt="e4m3")
    x = moe.layer(inp.x, *inp.weights, k=2, n_shared=1, logits=inp.logits, fmt=None)
    rel = np.abs(q["out_f64"] - x["out_f64"]).max(1) / np.abs(x["out_f64"]).max(1)
    assert rel.max() < 0.1


def test_zipf_generator_properties():
    cfg = synth.CONFIGS["skew32k"]
    lg = synth.gen_logits(cfg)
    ids, _ = moe.route_topk(lg, cfg.k)
    counts = np.bincount(ids.reshape(-1), minlength=cfg.E)
    assert (counts == 0).sum() >= 4
    assert (counts > 0.05 * ids.size).sum() >= 3
