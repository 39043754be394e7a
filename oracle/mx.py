"""Bit-level number formats used by the routed-expert path (fp64, numpy).

Test infrastructure: see the package docstring. Everything here is written
from the bit definitions, never from a lookup table shared with the GPU code.

Formats
-------
* Expert weights are FP4 e2m1 codes, two per byte, with one E8M0 scale per 32
  consecutive weights along the reduction axis (paper: Historical TP4 decode
  optimization / Parallel decomposition -- packed 4-bit FP4 weights, the e2m1
  nibble mapping to the doubled integers {0,+-1,+-2,+-3,+-4,+-6,+-8,+-12}, and
  E8M0 scaling; Correctness recovery / Later numerical and integration repairs
  -- logical E8M0 scales).
* Activations are quantised per block of 32 elements before each projection
  (paper: the same bullet list -- online activation quantisation per 32
  elements; Prefill optimization / From per-assignment scalar work to CDNA2
  MFMA -- native activation quantisation). The paper's gfx90a kernels used
  INT8; the gfx950 matrix cores take OCP microscaling (MX) element formats, so
  the element format here is one of e4m3 (MXFP8), e2m3 (MXFP6), e2m1 (MXFP4)
  with an E8M0 block scale.

Readings where the paper is silent:
* nibble order: element 2i sits in bits 0-3 of byte i, element 2i+1 in bits 4-7;
* E8M0 byte b decodes to 2**(b-127); b == 255 is NaN (OCP MX v1.0);
* the activation block scale is the smallest power of two 2**X that lets the
  block's largest magnitude fit under the element format's largest finite value
  (so no element saturates); X is clamped to [-127, 127]; an all-zero block gets
  X = 0 (byte 127);
* every element is rounded to nearest, ties to even, onto the element grid
  (subnormals included); the sign bit is the sign bit of the input, so -0.0 and
  negative values that round to zero keep the sign bit.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


# ---------------------------------------------------------------------------
# FP4 e2m1 weight codes and E8M0 scales
# ---------------------------------------------------------------------------

def e2m1_decode(codes) -> np.ndarray:
    """Decode 4-bit e2m1 codes (values 0..15) to fp64 from their bits.

    Bit 3 is the sign, bits 2..1 the exponent field (bias 1), bit 0 the
    mantissa. Exponent field 0 is subnormal: value 0.5*m. Otherwise the value
    is 2**(ef-1) * (1 + m/2). Pinned by the paper's doubled-integer nibble map
    (Historical TP4 decode optimization / Parallel decomposition): twice this
    table is {0, 1, 2, 3, 4, 6, 8, 12} and their negatives.
    """
    c = np.asarray(codes).astype(np.int64)
    if np.any((c < 0) | (c > 15)):
        raise ValueError("e2m1 code out of range")
    sign = np.where((c >> 3) & 1, -1.0, 1.0)
    ef = (c >> 1) & 3
    m = (c & 1).astype(np.float64)
    mag = np.where(ef == 0, 0.5 * m, np.ldexp(1.0 + 0.5 * m, ef - 1))
    return sign * mag


def unpack_nibbles(packed) -> np.ndarray:
    """Split packed bytes [..., K/2] into codes [..., K]; element 2i is the low nibble."""
    p = np.asarray(packed, dtype=np.uint8)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = p & 0x0F
    out[..., 1::2] = p >> 4
    return out


def pack_nibbles(codes) -> np.ndarray:
    """Inverse of :func:`unpack_nibbles` (codes [..., K] with K even)."""
    c = np.asarray(codes, dtype=np.uint8)
    if c.shape[-1] % 2:
        raise ValueError("need an even number of codes")
    return (c[..., 0::2] & 0x0F) | ((c[..., 1::2] & 0x0F) << 4)


def e8m0_decode(b) -> np.ndarray:
    """E8M0 scale byte -> fp64: 2**(b-127); byte 255 is NaN."""
    bb = np.asarray(b).astype(np.int64)
    if np.any((bb < 0) | (bb > 255)):
        raise ValueError("e8m0 byte out of range")
    v = np.ldexp(1.0, bb - 127)
    return np.where(bb == 255, np.nan, v)


def dequant_fp4(packed, scales) -> np.ndarray:
    """Dequantise one FP4 weight matrix.

    packed: uint8 [N, K/2] (two e2m1 codes per byte); scales: uint8 [N, K/32]
    (one E8M0 byte per 32 consecutive K elements). Returns fp64 [N, K] with
    W[n, kk] = e2m1(code[n, kk]) * e8m0(scales[n, kk // 32]) -- exact in fp64.
    The 16 code values are decoded from their bits once and looked up per
    code (the same values as decoding every code, in a fraction of the time).
    """
    vals = e2m1_decode(np.arange(16))[unpack_nibbles(packed)]
    s = e8m0_decode(scales)
    n, k = vals.shape
    if s.shape != (n, k // 32):
        raise ValueError(f"scale shape {s.shape} does not match weights {vals.shape}")
    return (vals.reshape(n, k // 32, 32) * s[:, :, None]).reshape(n, k)


# ---------------------------------------------------------------------------
# MX element formats for activations
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class ElemFormat:
    name: str
    ebits: int       # exponent field width
    mbits: int       # mantissa field width
    bias: int        # exponent bias
    nan_code: int    # magnitude code that is NaN (-1: none)

    @property
    def emin(self) -> int:
        """Exponent of the smallest normal value."""
        return 1 - self.bias

    @property
    def max_code(self) -> int:
        """Largest finite magnitude code."""
        top = (1 << (self.ebits + self.mbits)) - 1
        return top - 1 if self.nan_code == top else top

    @property
    def maxval(self) -> float:
        return float(elem_decode(np.array([self.max_code]), self)[0])

    @property
    def emax(self) -> int:
        """Exponent of the largest finite value."""
        return int(np.frexp(self.maxval)[1]) - 1

    @property
    def max_mant(self) -> float:
        """Significand (in [1, 2)) of the largest finite value."""
        return self.maxval / 2.0 ** self.emax

    @property
    def bits(self) -> int:
        return 1 + self.ebits + self.mbits


# OCP MX v1.0 element formats: e4m3 has no infinities and one NaN magnitude
# (all exponent and mantissa bits set); e2m3 and e2m1 have neither.
E4M3 = ElemFormat("e4m3", 4, 3, 7, 0x7F)
E2M3 = ElemFormat("e2m3", 2, 3, 1, -1)
E2M1 = ElemFormat("e2m1", 2, 1, 1, -1)
FORMATS = {"e4m3": E4M3, "e2m3": E2M3, "e2m1": E2M1}


def _fmt(f) -> ElemFormat:
    return FORMATS[f] if isinstance(f, str) else f


def elem_decode(codes, fmt) -> np.ndarray:
    """Decode element codes of an MX element format to fp64 from the bits."""
    f = _fmt(fmt)
    c = np.asarray(codes).astype(np.int64)
    nb = f.ebits + f.mbits
    sign = np.where((c >> nb) & 1, -1.0, 1.0)
    mag_code = c & ((1 << nb) - 1)
    ef = mag_code >> f.mbits
    m = (mag_code & ((1 << f.mbits) - 1)).astype(np.float64)
    frac = m / (1 << f.mbits)
    mag = np.where(ef == 0, np.ldexp(frac, f.emin), np.ldexp(1.0 + frac, ef - f.bias))
    if f.nan_code >= 0:
        mag = np.where(mag_code == f.nan_code, np.nan, mag)
    return sign * mag


def _round_to_elem(q: np.ndarray, f: ElemFormat) -> np.ndarray:
    """Round fp64 values to the nearest element code, ties to even."""
    neg = np.signbit(q)
    a = np.abs(q)
    _, ex = np.frexp(a)                  # a = mant * 2**ex, mant in [0.5, 1)
    e = np.where(a == 0, f.emin, np.maximum(ex - 1, f.emin))
    n = np.rint(np.ldexp(a, f.mbits - e))     # significand in units of 2**(e-mbits)
    carry = n >= (1 << (f.mbits + 1))         # rounded up into the next binade
    e = np.where(carry, e + 1, e)
    n = np.where(carry, n / 2, n)
    sub = (e == f.emin) & (n < (1 << f.mbits))
    ef = np.where(sub, 0, e - f.emin + 1)
    mf = np.where(sub, n, n - (1 << f.mbits)).astype(np.int64)
    mag_code = (ef.astype(np.int64) << f.mbits) | mf
    mag_code = np.minimum(mag_code, f.max_code)   # saturate (never hit with the scale rule)
    return ((neg.astype(np.int64) << (f.ebits + f.mbits)) | mag_code).astype(np.uint8)


def mx_scale_exponent(amax, fmt) -> np.ndarray:
    """Block scale exponent X for block maxima ``amax`` (fp64 array).

    X is the smallest integer with amax <= maxval * 2**X, clamped to
    [-127, 127]; amax == 0 gives X = 0. Writing amax = m * 2**f with m in
    [1, 2): X = f - emax when m <= max_mant, else f - emax + 1.
    """
    f = _fmt(fmt)
    amax = np.asarray(amax, dtype=np.float64)
    mant, ex = np.frexp(amax)
    m, fexp = 2.0 * mant, ex - 1
    x = np.where(m <= f.max_mant, fexp - f.emax, fexp - f.emax + 1)
    x = np.where(amax == 0, 0, x)
    return np.clip(x, -127, 127).astype(np.int64)


def mx_quantize(v, fmt):
    """Quantise fp64 values [..., K] (K % 32 == 0) per block of 32 along K.

    Returns (codes uint8 [..., K], one code per byte, and scale bytes uint8
    [..., K/32]). Element codes are RNE(v / 2**X) on the element grid with the
    block exponent X from :func:`mx_scale_exponent`.
    """
    f = _fmt(fmt)
    v = np.asarray(v, dtype=np.float64)
    k = v.shape[-1]
    if k % 32:
        raise ValueError("K must be a multiple of 32")
    blocks = v.reshape(v.shape[:-1] + (k // 32, 32))
    x = mx_scale_exponent(np.max(np.abs(blocks), axis=-1), f)
    q = np.ldexp(blocks, -x[..., None])
    codes = _round_to_elem(q, f).reshape(v.shape)
    return codes, (x + 127).astype(np.uint8)


def mx_dequantize(codes, scale_bytes, fmt) -> np.ndarray:
    """Inverse map of :func:`mx_quantize`: element value * 2**(byte-127)."""
    f = _fmt(fmt)
    vals = elem_decode(codes, f)
    k = vals.shape[-1]
    s = e8m0_decode(scale_bytes)
    return (vals.reshape(vals.shape[:-1] + (k // 32, 32)) * s[..., None]).reshape(vals.shape)


# ---------------------------------------------------------------------------
# bf16
# ---------------------------------------------------------------------------

def bf16_to_f64(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> fp64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    with np.errstate(invalid="ignore"):          # signalling-NaN patterns
        return b.view(np.float32).astype(np.float64)


def f64_to_bf16(v) -> np.ndarray:
    """Round fp64 to bf16 (round to nearest, ties to even), returned as uint16 bits.

    bf16 keeps 8 significant bits; its smallest normal is 2**-126 and its
    subnormal quantum 2**-133. Values beyond the largest finite bf16 after
    rounding become infinities; NaN stays NaN.
    """
    v = np.asarray(v, dtype=np.float64)
    _, ex = np.frexp(v)
    ex = np.maximum(ex, -125)
    q = np.rint(np.ldexp(v, 8 - ex))
    with np.errstate(over="ignore"):
        r = np.ldexp(q, ex - 8).astype(np.float32)   # exact unless it overflows to inf
    return (r.view(np.uint32) >> 16).astype(np.uint16)
