"""Pins of the oracle's number formats (CPU only).

Each test ties oracle/mx.py to something other than itself: the paper's
printed nibble map, PyTorch's float8/bfloat16 conversions, or an exhaustive
brute-force nearest-code search written independently in tests/bruteforce.py.
"""
import fractions
import math

import numpy as np
import pytest
import torch

from oracle import mx
from tests import bruteforce as bf


def test_e2m1_matches_paper_doubled_map():
    """2x the e2m1 table is the paper's nibble map {0,+-1,+-2,+-3,+-4,+-6,+-8,+-12}."""
    ours = mx.e2m1_decode(np.arange(16))
    paper = np.array(bf.paper_e2m1_table())
    assert np.array_equal(ours, paper)
    assert np.array_equal(np.signbit(ours), np.signbit(paper))   # -0 for code 8
    assert sorted(set(np.abs(2 * ours).astype(int))) == [0, 1, 2, 3, 4, 6, 8, 12]


def test_e2m1_roundtrip_all_codes():
    """encode(decode(c)) == c for all 16 codes, including -0 -> 8."""
    vals = mx.e2m1_decode(np.arange(16))
    codes = mx._round_to_elem(vals, mx.E2M1)
    assert np.array_equal(codes, np.arange(16))
    assert np.array_equal(mx.elem_decode(np.arange(16), "e2m1"), vals)


def test_nibble_order_low_first():
    codes = np.array([[1, 2, 15, 0]], np.uint8)
    packed = mx.pack_nibbles(codes)
    assert packed.tolist() == [[0x21, 0x0F]]
    assert np.array_equal(mx.unpack_nibbles(packed), codes)


def test_nibble_fingerprint_single_weight():
    """A single nonzero weight at a known K index shows up at exactly that index."""
    for kk in (0, 1, 31, 32, 63):
        codes = np.zeros((1, 64), np.uint8)
        codes[0, kk] = 7                                # value 6.0
        scales = np.array([[127, 129]], np.uint8)       # 1.0 and 4.0
        w = mx.dequant_fp4(mx.pack_nibbles(codes), scales)
        expect = np.zeros((1, 64))
        expect[0, kk] = 6.0 * (1.0 if kk < 32 else 4.0)
        assert np.array_equal(w, expect)


def test_e8m0_decode():
    b = np.array([0, 1, 126, 127, 128, 254, 255])
    v = mx.e8m0_decode(b)
    assert v[0] == 2.0 ** -127 and v[1] == 2.0 ** -126
    assert v[2] == 0.5 and v[3] == 1.0 and v[4] == 2.0 and v[5] == 2.0 ** 127
    assert np.isnan(v[6])


def test_e4m3_decode_matches_torch_all_codes():
    """Every e4m3 code decodes as torch.float8_e4m3fn does (OCP e4m3, NaN 0x7F/0xFF)."""
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = mx.elem_decode(codes, "e4m3")
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(ours))
    assert np.array_equal(ours[~nan], ref[~nan])
    assert mx.E4M3.maxval == 448.0 and mx.E4M3.emax == 8 and mx.E4M3.max_mant == 1.75


@pytest.mark.parametrize("fmt", ["e4m3", "e2m3", "e2m1"])
def test_elem_decode_matches_enumeration(fmt):
    ours = mx.elem_decode(np.arange(2 ** mx.FORMATS[fmt].bits), fmt)
    ref = bf.table(fmt)
    for c, (a, b) in enumerate(zip(ours, ref)):
        if b is None:
            assert np.isnan(a), c
        else:
            assert a == b and math.copysign(1, a) == math.copysign(1, b), c


@pytest.mark.parametrize("fmt,maxval,emax,mm", [("e4m3", 448, 8, 1.75), ("e2m3", 7.5, 2, 1.875),
                                                ("e2m1", 6.0, 2, 1.5)])
def test_format_extremes(fmt, maxval, emax, mm):
    f = mx.FORMATS[fmt]
    assert (f.maxval, f.emax, f.max_mant) == (maxval, emax, mm)


def _all_finite_bf16():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = mx.bf16_to_f64(bits)
    return v[np.isfinite(v)]


@pytest.mark.parametrize("fmt", ["e4m3", "e2m3", "e2m1"])
def test_scale_exponent_brute_force(fmt):
    """Block exponent = smallest X with amax <= max * 2**X, over every positive bf16."""
    v = _all_finite_bf16()
    v = np.unique(np.abs(v))
    rng = np.random.default_rng(1)
    pick = np.concatenate([v[:50], v[-50:], rng.choice(v, 600, replace=False)])
    ours = mx.mx_scale_exponent(pick, fmt)
    for a, x in zip(pick, ours):
        assert x == bf.block_scale_exponent(float(a), fmt), (a, x)


def _nearest_codes_vectorised(q, fmt):
    """Brute force over all codes at once; ties to the even code; sign of q kept."""
    tab = bf.table(fmt)
    half = len(tab) // 2
    mags = np.array([np.inf if t is None else t for t in tab[:half]])
    d = np.abs(np.abs(q)[:, None] - mags[None, :])
    dmin = d.min(axis=1, keepdims=True)
    cand = d == dmin
    even = cand & (np.arange(half)[None, :] % 2 == 0)
    pick = np.where(even.any(axis=1), even.argmax(axis=1), cand.argmax(axis=1))
    return (pick + np.where(np.signbit(q), half, 0)).astype(np.uint8)


@pytest.mark.parametrize("fmt", ["e4m3", "e2m3", "e2m1"])
@pytest.mark.parametrize("x0", [0, -9, 20, -126, 100])
def test_quantize_exhaustive_bf16(fmt, x0):
    """Every finite bf16 v with |v| <= max*2**x0, in a block whose maximum fixes
    the exponent at x0, quantises to the brute-force nearest code of v/2**x0."""
    f = mx.FORMATS[fmt]
    cap = f.maxval * 2.0 ** x0
    v = _all_finite_bf16()
    v = v[np.abs(v) <= cap]
    n = v.size
    nb = -(-n // 31)
    blocks = np.zeros((nb, 32))
    flat = np.zeros(nb * 31)
    flat[:n] = v
    blocks[:, 1:] = flat.reshape(nb, 31)
    blocks[:, 0] = cap                       # companion lane fixes the exponent
    codes, sb = mx.mx_quantize(blocks, fmt)
    assert np.all(sb == x0 + 127)
    got = codes[:, 1:].reshape(-1)[:n]
    want = _nearest_codes_vectorised(np.ldexp(v, -x0), fmt)
    assert np.array_equal(got, want)


def test_quantize_matches_torch_e4m3_cast():
    """Element rounding equals PyTorch's fp32 -> float8_e4m3fn cast (RNE) in range."""
    rng = np.random.default_rng(2)
    v = (rng.standard_normal((512, 256)) * np.exp(rng.uniform(-20, 20, (512, 1)))).astype(np.float32)
    codes, sb = mx.mx_quantize(v.astype(np.float64), "e4m3")
    x = sb.astype(np.int64) - 127
    q = np.ldexp(v.astype(np.float64).reshape(512, 8, 32), -x[..., None]).astype(np.float32)
    ref = torch.from_numpy(q.reshape(512, 256)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes, ref)


def test_quantize_zero_block_and_h1_value():
    codes, sb = mx.mx_quantize(np.zeros((1, 32)), "e4m3")
    assert sb.tolist() == [[127]] and not codes.any()
    h = 256.0 / (1.0 + math.exp(-16.0))
    codes, sb = mx.mx_quantize(np.full((1, 32), h), "e4m3")
    assert sb.tolist() == [[127]]
    assert np.all(mx.mx_dequantize(codes, sb, "e4m3") == 256.0)


def test_bf16_roundtrip_and_torch_rounding():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = mx.bf16_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    fin = np.isfinite(ref)
    assert np.array_equal(v[fin], ref[fin])
    back = mx.f64_to_bf16(v[fin])
    assert np.array_equal(back, bits[fin])
    rng = np.random.default_rng(3)
    f = (rng.standard_normal(100000) * np.exp(rng.uniform(-80, 80, 100000))).astype(np.float32)
    want = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mx.f64_to_bf16(f.astype(np.float64)), want)


def test_bf16_rounding_of_fp64_exact():
    """fp64 inputs (not fp32-representable) round to the nearest bf16, ties to even,
    checked with exact rational arithmetic."""
    rng = np.random.default_rng(4)
    v = rng.standard_normal(300) * np.exp(rng.uniform(-30, 30, 300))
    mids = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8)])
    v = np.concatenate([v, mids])
    got = mx.bf16_to_f64(mx.f64_to_bf16(v))
    for a, g in zip(v, got):
        fa = fractions.Fraction(float(a))
        _, ex = math.frexp(a)
        q = fractions.Fraction(2) ** (ex - 8)
        lo = (fa / q).__floor__() * q
        hi = lo + q
        dlo, dhi = fa - lo, hi - fa
        if dlo < dhi:
            want = lo
        elif dhi < dlo:
            want = hi
        else:
            want = lo if (lo / q) % 2 == 0 else hi
        assert fractions.Fraction(float(g)) == want, a
