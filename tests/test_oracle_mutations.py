"""Plant plausible mistakes in the oracle (on the CPU) and check the pins catch each.

Every mutation below replaces one oracle function with a subtly wrong copy; the
pin battery (the same checks as test_oracle_formats / test_oracle_layer, in
condensed form) must fail for every one of them. This shows the pins are
discriminating, not just self-consistent.
"""
import contextlib
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


def _const(h, i, w2_scale=127):
    b = 2 | (2 << 4)
    return (np.full((2 * i, h // 2), b, np.uint8), np.full((2 * i, h // 32), 127, np.uint8),
            np.full((h, i // 2), b, np.uint8), np.full((h, i // 32), w2_scale, np.uint8))


def _pins():
    """Run the condensed pin battery; return the names of the pins that fail."""
    bad = []

    def check(name, fn):
        try:
            ok = fn()
        except Exception:
            ok = False
        if not ok:
            bad.append(name)

    check("paper_e2m1", lambda: np.array_equal(mx.e2m1_decode(np.arange(16)),
                                               np.array(bf.paper_e2m1_table())))
    check("e8m0", lambda: mx.e8m0_decode(np.array([127, 128]))[1] == 2.0
          and mx.e8m0_decode(np.array([127]))[0] == 1.0)

    x = np.full((1, 32), 0x3F00, np.uint16)
    w1 = tuple(np.stack([a]) for a in _const(32, 32))
    check("H1", lambda: np.all(moe.layer(x, *w1, k=1, logits=np.zeros((1, 1), np.float32))
                               ["out_f64"] == HAND["H1"]["out"]))
    e0, e2 = _const(32, 32), _const(32, 32, 128)
    w4 = tuple(np.stack(z) for z in zip(e0, e0, e2, e0))
    check("H2", lambda: np.all(moe.layer(x, *w4, k=2, logits=np.array([[1, 3, 3, 0]], np.float32))
                               ["out_f64"] == HAND["H2"]["out"]))
    h3 = HAND["H3"]
    check("H3", lambda: moe.permute(np.array(h3["ids"]), 3)[2].tolist() == h3["sorted"])
    check("ties", lambda: moe.route_topk(np.array([[0.5, 2, 2, -1, 2]], np.float32), 3)[0]
          .tolist() == [[1, 2, 4]])
    lg = np.random.default_rng(0).standard_normal((8, 6)).astype(np.float32)

    def soft():
        ids, w = moe.route_topk(lg, 6)
        return np.allclose(np.take_along_axis(scipy.special.softmax(lg.astype(float), 1), ids, 1), w)
    check("softmax", soft)

    def renorm():
        _, w = moe.route_topk(lg, 2)
        return np.allclose(w.sum(1), 1.0)
    check("renorm", renorm)

    def quant():
        v = np.linspace(-448, 448, 31 * 64)
        blocks = np.concatenate([np.full((64, 1), 448.0), v.reshape(64, 31)], 1)
        codes, _ = mx.mx_quantize(blocks, "e4m3")
        want = np.array([bf.nearest_code(float(q), "e4m3") for q in blocks.reshape(-1)])
        return np.array_equal(codes.reshape(-1), want)
    check("quant", quant)

    def scale_rule():
        return all(mx.mx_scale_exponent(a, "e4m3") == bf.block_scale_exponent(a, "e4m3")
                   for a in (0.5, 255.99997, 1.0, 448.0, 449.0, 3e-5))
    check("scale_rule", scale_rule)

    h4 = HAND["H4"]
    x4 = np.array(h4["x_bits"], np.uint16)
    wr4 = np.repeat(np.array(h4["wr_row_bits"], np.uint16)[:, None], x4.shape[1], axis=1)
    check("H4", lambda: moe.router_logits(x4, wr4).tolist() == h4["logits"])

    def router_brute():
        rng = np.random.default_rng(3)
        xb = synth.f32_to_bf16_bits(rng.standard_normal((3, 40)).astype(np.float32))
        wb = synth.f32_to_bf16_bits(rng.standard_normal((5, 40)).astype(np.float32))
        ref = np.array(bf.router_logits(xb.tolist(), wb.tolist()))
        return np.all(np.abs(moe.router_logits(xb, wb) - ref) <= 1e-14 * np.abs(ref).max())
    check("router_brute", router_brute)

    def brute():
        cfg = synth.LayerConfig("mut", 3, 64, 4, 2, 64, 1, "normal", 21)
        inp = synth.make_inputs(cfg)
        r = moe.layer(inp.x, *inp.weights, k=2, n_shared=1, logits=inp.logits)
        ref = np.array(bf.layer(mx.bf16_to_f64(inp.x).tolist(), inp.logits.astype(float).tolist(),
                                *(a.tolist() for a in inp.weights), 2, 1, "e4m3"))
        return np.all(np.abs(r["out_f64"] - ref) <= 1e-12 * np.abs(ref).max(1, keepdims=True))
    check("brute", brute)
    return bad


@contextlib.contextmanager
def patched(mod, name, fn):
    old = getattr(mod, name)
    setattr(mod, name, fn)
    try:
        yield
    finally:
        setattr(mod, name, old)


_orig = {n: getattr(moe, n) for n in ("router_logits", "route_topk", "permute", "swiglu",
                                      "expert_ffn", "combine")}
_origmx = {n: getattr(mx, n) for n in ("e2m1_decode", "e8m0_decode", "unpack_nibbles",
                                       "mx_scale_exponent", "_round_to_elem", "dequant_fp4")}


def m_router_transposed(x_bits, wr_bits):
    """Router matrix read as [H, E] (its buffer reinterpreted) instead of [E, H]."""
    wr = mx.bf16_to_f64(wr_bits)
    return mx.bf16_to_f64(x_bits) @ wr.reshape(wr.shape[1], wr.shape[0])


def m_router_fp32(x_bits, wr_bits):
    """x and the router weights cast to fp32 before the product (fp32 sums)."""
    x32 = mx.bf16_to_f64(x_bits).astype(np.float32)
    w32 = mx.bf16_to_f64(wr_bits).astype(np.float32)
    return (x32 @ w32.T).astype(np.float64)


def m_swiglu_sign(g, u):
    with np.errstate(over="ignore"):
        return g * u / (1.0 + np.exp(g))


def m_swiglu_gate_only(g, u):
    return _orig["swiglu"](g, np.ones_like(u))


def m_route_ties_high(logits, k, n_shared=0):
    lg = np.asarray(logits)[:, ::-1]
    ids, w = _orig["route_topk"](lg, k, n_shared)
    e = lg.shape[1]
    ids = ids.copy()
    ids[:, :k] = e - 1 - ids[:, :k]
    return ids, w


def m_route_no_renorm(logits, k, n_shared=0):
    ids, w = _orig["route_topk"](logits, k, n_shared)
    full = scipy.special.softmax(np.asarray(logits, float), 1)
    w = w.copy()
    w[:, :k] = np.take_along_axis(full, ids[:, :k], 1)
    return ids, w


def m_permute_unstable(ids, ne):
    counts, offsets, srt, pos = _orig["permute"](ids, ne)
    srt = srt.copy()
    for e in range(ne):
        srt[offsets[e]:offsets[e + 1]] = srt[offsets[e]:offsets[e + 1]][::-1]
    pos = np.empty_like(srt)
    pos[srt] = np.arange(srt.size)
    return counts, offsets, srt, pos


def m_ffn_swap_gate_up(a, w13, w13s, w2, w2s, fmt):
    i = w13.shape[0] // 2
    sw = lambda z: np.concatenate([z[i:], z[:i]])   # noqa: E731
    return _orig["expert_ffn"](a, sw(w13), sw(w13s), w2, w2s, fmt)


def m_ffn_w2_transposed(a, w13, w13s, w2, w2s, fmt):
    codes = mx.unpack_nibbles(w2)
    if codes.shape[0] != codes.shape[1]:
        return _orig["expert_ffn"](a, w13, w13s, w2, w2s, fmt)
    vals = mx.dequant_fp4(w2, w2s).T          # transposed operand
    r = _orig["expert_ffn"](a, w13, w13s, w2, w2s, fmt)
    r["p"] = r["hd"] @ vals.T
    return r


def m_combine_drop_last(p, w):
    w = np.asarray(w, float).copy()
    w[:, -1] = 0
    return _orig["combine"](p, w)


def m_combine_square_w(p, w):
    return _orig["combine"](p, np.asarray(w, float) ** 2)


def m_e2m1_subnormal(codes):
    c = np.asarray(codes).astype(np.int64)
    v = _origmx["e2m1_decode"](c)
    return np.where(((c >> 1) & 3) == 0, 2 * v, v)


def m_e8m0_bias(b):
    return _origmx["e8m0_decode"](b) / 2


def m_nibbles_high_first(p):
    out = _origmx["unpack_nibbles"](p)
    out2 = out.copy()
    out2[..., 0::2], out2[..., 1::2] = out[..., 1::2], out[..., 0::2]
    return out2


def m_scale_floor(amax, fmt):
    f = mx._fmt(fmt)
    mant, ex = np.frexp(np.asarray(amax, float))
    x = np.where(np.asarray(amax) == 0, 0, ex - 1 - f.emax)
    return np.clip(x, -127, 127).astype(np.int64)


def m_round_truncate(q, f):
    a = np.abs(q)
    _, ex = np.frexp(a)
    e = np.where(a == 0, f.emin, np.maximum(ex - 1, f.emin))
    step = np.ldexp(1.0, e - f.mbits)
    return _origmx["_round_to_elem"](np.sign(q) * np.floor(a / step) * step, f)


def m_scale_index_off(packed, scales):
    return _origmx["dequant_fp4"](packed, np.roll(scales, 1, axis=1))


MUTATIONS = {
    "router_transposed": (moe, "router_logits", m_router_transposed),
    "router_fp32": (moe, "router_logits", m_router_fp32),
    "swiglu_sign": (moe, "swiglu", m_swiglu_sign),
    "swiglu_drops_up": (moe, "swiglu", m_swiglu_gate_only),
    "route_ties_high": (moe, "route_topk", m_route_ties_high),
    "route_no_renorm": (moe, "route_topk", m_route_no_renorm),
    "permute_unstable": (moe, "permute", m_permute_unstable),
    "ffn_swap_gate_up": (moe, "expert_ffn", m_ffn_swap_gate_up),
    "ffn_w2_transposed": (moe, "expert_ffn", m_ffn_w2_transposed),
    "combine_drops_shared": (moe, "combine", m_combine_drop_last),
    "combine_squares_w": (moe, "combine", m_combine_square_w),
    "e2m1_subnormal": (mx, "e2m1_decode", m_e2m1_subnormal),
    "e8m0_bias": (mx, "e8m0_decode", m_e8m0_bias),
    "nibbles_high_first": (mx, "unpack_nibbles", m_nibbles_high_first),
    "scale_floor_rule": (mx, "mx_scale_exponent", m_scale_floor),
    "round_truncate": (mx, "_round_to_elem", m_round_truncate),
    "scale_index_off": (mx, "dequant_fp4", m_scale_index_off),
}


def test_unmutated_oracle_passes_battery():
    assert _pins() == []


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name):
    mod, attr, fn = MUTATIONS[name]
    with patched(mod, attr, fn):
        failed = _pins()
    assert failed, f"mutation {name} slipped past every pin"
