"""Pure-Python brute force used to pin the fp64 oracle on tiny inputs.

Independent of ``oracle/``: its FP4 values come from the paper's printed
doubled-integer nibble map (tests/golden/e2m1_doubled_map.txt), element
formats are enumerated code by code, quantisation picks the nearest code by
exhaustive search (ties to the even code), the block scale is found by
counting up from the smallest exponent, and every sum is an explicit loop.
"""
from __future__ import annotations

import math
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def paper_e2m1_table():
    """code -> value, from the paper's doubled map divided by 2."""
    tab = {}
    with open(os.path.join(GOLDEN, "e2m1_doubled_map.txt")) as f:
        for line in f:
            line = line.split("#")[0].split()
            if len(line) == 2:
                code, dbl = int(line[0]), float(line[1])
                tab[code] = dbl / 2.0
    assert len(tab) == 16
    return [tab[c] for c in range(16)]


def enumerate_format(ebits, mbits, bias, nan_magnitude=None):
    """All codes of a sign/exponent/mantissa format -> value (None for NaN)."""
    vals = []
    nmag = 1 << (ebits + mbits)
    for code in range(2 * nmag):
        sign = -1.0 if code >= nmag else 1.0
        mag = code % nmag
        if nan_magnitude is not None and mag == nan_magnitude:
            vals.append(None)
            continue
        e = mag >> mbits
        m = mag & ((1 << mbits) - 1)
        if e == 0:
            v = (m / (1 << mbits)) * 2.0 ** (1 - bias)
        else:
            v = (1 + m / (1 << mbits)) * 2.0 ** (e - bias)
        vals.append(sign * v)
    return vals


FORMAT_TABLES = {
    "e4m3": enumerate_format(4, 3, 7, nan_magnitude=0x7F),
    "e2m3": enumerate_format(2, 3, 1),
    "e2m1": None,  # filled lazily from the paper's map
}


def table(fmt):
    if fmt == "e2m1":
        return paper_e2m1_table()
    return FORMAT_TABLES[fmt]


def nearest_code(q, fmt):
    """Code whose value is nearest to q; ties go to the code with an even mantissa
    (code LSB 0). The sign bit follows the sign of q (so -0.0 keeps it)."""
    tab = table(fmt)
    half = len(tab) // 2
    neg = math.copysign(1.0, q) < 0
    a = abs(q)
    best, bestd = None, None
    for code in range(half):            # magnitudes only
        v = tab[code]
        if v is None:
            continue
        d = abs(a - v)
        if bestd is None or d < bestd or (d == bestd and code % 2 == 0 and best % 2 == 1):
            best, bestd = code, d
    return best + (half if neg else 0)


def max_finite(fmt):
    return max(v for v in table(fmt) if v is not None)


def block_scale_exponent(amax, fmt):
    """Smallest X in [-127, 127] with amax <= max_finite * 2**X (0 for amax == 0)."""
    if amax == 0:
        return 0
    mx = max_finite(fmt)
    for x in range(-127, 128):
        if amax <= mx * 2.0 ** x:
            return x
    return 127


def quantize_block(vals, fmt):
    """One block of 32 -> (codes, scale byte, dequantised values)."""
    amax = max(abs(v) for v in vals)
    x = block_scale_exponent(amax, fmt)
    codes = [nearest_code(v / 2.0 ** x, fmt) for v in vals]
    tab = table(fmt)
    deq = [tab[c] * 2.0 ** x for c in codes]
    return codes, x + 127, deq


def quantize_row(vals, fmt):
    codes, scales, deq = [], [], []
    for b in range(0, len(vals), 32):
        c, s, d = quantize_block(vals[b:b + 32], fmt)
        codes += c
        scales.append(s)
        deq += d
    return codes, scales, deq


def round_bf16(v):
    """Nearest bf16 value (8 significant bits, ties to the even significand) of
    a finite float in the normal bf16 range, by Python's round-half-even."""
    if v == 0:
        return v
    m, e = math.frexp(v)                   # v = m * 2**e, 0.5 <= |m| < 1
    return round(m * 256) * 2.0 ** (e - 8)


def dequant_weight(packed_row, scale_row):
    """One weight row: packed bytes (low nibble first) and E8M0 bytes -> values."""
    tab = paper_e2m1_table()
    out = []
    for i, byte in enumerate(packed_row):
        for code in (byte & 15, byte >> 4):
            kk = len(out)
            out.append(tab[code] * 2.0 ** (scale_row[kk // 32] - 127))
    return out


def bf16_value(bits):
    """A bf16 bit pattern (normal or zero) -> its value, from the fields."""
    sign = -1.0 if bits >> 15 else 1.0
    ef, mf = (bits >> 7) & 0xFF, bits & 0x7F
    if ef == 0:
        return sign * mf * 2.0 ** -133
    return sign * (1 + mf / 128.0) * 2.0 ** (ef - 127)


def router_logits(x_bits, wr_bits):
    """logits[t][e] = sum_h x[t][h] * Wr[e][h] by explicit loops over bf16 bit
    patterns; math.fsum gives the exactly rounded sum of the exact products."""
    return [[math.fsum(bf16_value(a) * bf16_value(b) for a, b in zip(xr, wr)) for wr in wr_bits]
            for xr in x_bits]


def layer(x, logits, w13, w13s, w2, w2s, k, n_shared, fmt):
    """The routed layer by explicit loops (lists of Python floats).

    x: [T][H] floats; logits: [T][E]; w13[e]: [2I][H/2] bytes, w13s[e]: [2I][H/32],
    w2[e]: [H][I/2], w2s[e]: [H][I/32]. fmt None: no activation quantisation;
    'bf16': x unquantised, h rounded to bf16.
    Returns out [T][H] (unrounded floats).
    """
    T, H = len(x), len(x[0])
    E = len(logits[0])
    out = []
    for t in range(T):
        # top-k: repeatedly take the largest remaining logit, lower id on ties
        chosen = []
        for _ in range(k):
            best = None
            for e in range(E):
                if e in chosen:
                    continue
                if best is None or logits[t][e] > logits[t][best]:
                    best = e
            chosen.append(best)
        z = [math.exp(logits[t][e] - logits[t][chosen[0]]) for e in chosen]
        tot = sum(z)
        weights = [v / tot for v in z]
        experts = chosen + ([E] if n_shared else [])
        weights = weights + ([1.0] if n_shared else [])
        xa = quantize_row(x[t], fmt)[2] if fmt and fmt != "bf16" else list(x[t])
        acc = [0.0] * H
        for e, wt in zip(experts, weights):
            I = len(w13[e]) // 2
            w13d = [dequant_weight(w13[e][n], w13s[e][n]) for n in range(2 * I)]
            g = [sum(xa[hh] * w13d[n][hh] for hh in range(H)) for n in range(I)]
            u = [sum(xa[hh] * w13d[I + n][hh] for hh in range(H)) for n in range(I)]
            h = []
            for n in range(I):
                sig = 1.0 / (1.0 + math.exp(-g[n])) if g[n] > -700 else 0.0
                h.append(g[n] * sig * u[n])
            if fmt == "bf16":
                ha = [round_bf16(v) for v in h]
            else:
                ha = quantize_row(h, fmt)[2] if fmt else h
            for n in range(H):
                w2d = dequant_weight(w2[e][n], w2s[e][n])
                acc[n] += wt * sum(ha[i] * w2d[i] for i in range(I))
        out.append(acc)
    return out
