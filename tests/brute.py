"""Brute-force re-derivations used to pin the oracle on tiny inputs.

These share no code with the oracle: selection is by counting ranks,
quantization is exact rational arithmetic rounded to float32 by hand, and
attention is a scalar loop over keys with math.exp.  Only tiny inputs.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np


def bf16_value(bits) -> float:
    """bf16 bit pattern -> Python float (exact), by decoding the fields."""
    b = int(bits) & 0xFFFF
    sign = -1.0 if b >> 15 else 1.0
    e = (b >> 7) & 0xFF
    m = b & 0x7F
    if e == 0:
        return sign * m * 2.0 ** (-133)            # subnormal: m * 2^-7 * 2^-126
    if e == 0xFF:
        raise ValueError("inf/nan not expected")
    return sign * (1.0 + m / 128.0) * 2.0 ** (e - 127)


def round_to_f32(x: Fraction) -> Fraction:
    """Correctly round an exact rational to the nearest float32 (ties to even)."""
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = math.floor(math.log2(a.numerator) - math.log2(a.denominator))
    # fix possible off-by-one from the float log
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)                                # subnormal range shares the 2^-149 grid
    ulp = Fraction(2) ** (e - 23)
    q, r = divmod(a, ulp)
    q = int(q)
    if r > ulp / 2 or (r == ulp / 2 and q % 2 == 1):
        q += 1
    val = q * ulp
    if val >= Fraction(2) ** 128:
        raise OverflowError
    return sign * val


def round_half_even(x: Fraction) -> int:
    fl = math.floor(x)
    r = x - fl
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and fl % 2 == 1):
        return fl + 1
    return fl


def quant_block_exact(vals, c: int):
    """Symmetric block quantization with exact rationals: s = fl32(amax/c),
    code = clamp(rint(fl32(x/s)), -c, c).  ``vals`` are float32-exact numbers."""
    fr = [Fraction(float(v)) for v in vals]
    amax = max(abs(v) for v in fr)
    s = round_to_f32(amax / c)
    if s == 0:
        return [0] * len(fr), 0.0
    codes = [max(-c, min(c, round_half_even(round_to_f32(v / s)))) for v in fr]
    return codes, float(s)


def e4m3_value_exact(code: int) -> Fraction:
    """OCP FP8 E4M3 code -> exact rational, decoded from its fields (NaN codes
    raise).  Written from the format definition, independently of the oracle."""
    code = int(code) & 0xFF
    sign = -1 if code >> 7 else 1
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        raise ValueError("NaN code")
    if e == 0:
        return sign * Fraction(m, 8) * Fraction(1, 64)
    return sign * (1 + Fraction(m, 8)) * Fraction(2) ** (e - 7)


def e4m3_nearest(x: Fraction, negative: bool) -> int:
    """Nearest finite E4M3 code to the exact value x by enumeration (ties to
    the even code; beyond +-448 the nearest is +-448); the sign bit follows
    ``negative`` (so a negative input that rounds to zero gives 0x80)."""
    a = abs(x)
    best, bd = None, None
    for code in range(127):                       # non-negative finite codes
        d = abs(e4m3_value_exact(code) - a)
        if bd is None or d < bd or (d == bd and code % 2 == 0 and best % 2 == 1):
            best, bd = code, d
    return best | (0x80 if negative else 0)


def quant_block_fp8_exact(vals):
    """FP8 block quantization with exact rationals: s = fl32(amax/448),
    code = nearest E4M3 to fl32(x/s)."""
    fr = [Fraction(float(v)) for v in vals]
    amax = max(abs(v) for v in fr)
    s = round_to_f32(amax / 448)
    if s == 0:
        return [0] * len(fr), 0.0
    codes = []
    for v, raw in zip(fr, vals):
        y = round_to_f32(v / s)
        negative = y < 0 or (y == 0 and math.copysign(1.0, float(raw)) < 0)
        codes.append(e4m3_nearest(y, negative))
    return codes, float(s)


def e2m1_value_exact(code: int) -> Fraction:
    """OCP FP4 E2M1 code -> exact rational, from its fields: sign bit 3,
    exponent bits 2..1 with bias 1, mantissa bit 0; exponent 0 is subnormal.
    Written from the format definition, independently of the oracle."""
    code = int(code) & 0xF
    sign = -1 if code >> 3 else 1
    e = (code >> 1) & 0x3
    m = code & 0x1
    if e == 0:
        return sign * Fraction(m, 2)
    return sign * (1 + Fraction(m, 2)) * Fraction(2) ** (e - 1)


def e2m1_nearest(x: Fraction, negative: bool) -> int:
    """Nearest E2M1 code to the exact value x by enumeration (ties to the even
    code; beyond +-6 the nearest is +-6); sign bit from ``negative``."""
    a = abs(x)
    best, bd = None, None
    for code in range(8):
        d = abs(e2m1_value_exact(code) - a)
        if bd is None or d < bd or (d == bd and code % 2 == 0 and best % 2 == 1):
            best, bd = code, d
    return best | (0x8 if negative else 0)


def quant_block_fp4_exact(vals):
    """FP4 block quantization with exact rationals: s = fl32(amax/6), code =
    nearest E2M1 to fl32(x/s)."""
    fr = [Fraction(float(v)) for v in vals]
    amax = max(abs(v) for v in fr)
    s = round_to_f32(amax / 6)
    if s == 0:
        return [0] * len(fr), 0.0
    codes = []
    for v, raw in zip(fr, vals):
        y = round_to_f32(v / s)
        negative = y < 0 or (y == 0 and math.copysign(1.0, float(raw)) < 0)
        codes.append(e2m1_nearest(y, negative))
    return codes, float(s)


def e2m3_value_exact(code: int) -> Fraction:
    """OCP FP6 E2M3 code -> exact rational, from its fields: sign bit 5,
    exponent bits 4..3 with bias 1, mantissa bits 2..0; exponent 0 is
    subnormal.  Written from the format definition, independently of the
    oracle."""
    code = int(code) & 0x3F
    sign = -1 if code >> 5 else 1
    e = (code >> 3) & 0x3
    m = code & 0x7
    if e == 0:
        return sign * Fraction(m, 8)
    return sign * (1 + Fraction(m, 8)) * Fraction(2) ** (e - 1)


def e2m3_nearest(x: Fraction, negative: bool) -> int:
    """Nearest E2M3 code to the exact value x by enumeration of all 32
    magnitudes (ties to the even code; beyond +-7.5 the nearest is +-7.5);
    sign bit from ``negative``."""
    a = abs(x)
    best, bd = None, None
    for code in range(32):
        d = abs(e2m3_value_exact(code) - a)
        if bd is None or d < bd or (d == bd and code % 2 == 0 and best % 2 == 1):
            best, bd = code, d
    return best | (0x20 if negative else 0)


def quant_block_fp6_exact(vals):
    """FP6 block quantization with exact rationals: s = fl32(amax/7.5), code =
    nearest E2M3 to fl32(x/s)."""
    fr = [Fraction(float(v)) for v in vals]
    amax = max(abs(v) for v in fr)
    s = round_to_f32(amax / Fraction(15, 2))
    if s == 0:
        return [0] * len(fr), 0.0
    codes = []
    for v, raw in zip(fr, vals):
        y = round_to_f32(v / s)
        negative = y < 0 or (y == 0 and math.copysign(1.0, float(raw)) < 0)
        codes.append(e2m3_nearest(y, negative))
    return codes, float(s)


def topk_by_rank(S, k: int):
    """Position p is chosen iff fewer than k positions beat it, where p' beats p
    when S[p'] > S[p], or S[p'] == S[p] and p' < p.  Ascending output."""
    S = [float(v) for v in S]          # -0.0 == 0.0 in Python comparisons
    chosen = []
    for p in range(len(S)):
        beat = sum(1 for q in range(len(S)) if S[q] > S[p] or (S[q] == S[p] and q < p))
        if beat < k:
            chosen.append(p)
    return chosen


def attention_rows(Qv, Kv, Vv, L, W, bits, block, idx_list, qcodes, qscales,
                   kcodes, kscales, vcodes, vscales, fp8: bool = False, band: bool = False,
                   fp4: bool = False, q6: bool = False):
    """Scalar-loop hybrid attention for one (batch, head).

    band: the per-query window (row t sees keys t+1-W .. t in full precision,
    a quantizable key only quantized when it is older than that).
    fp8: every code is E4M3; fp4: Q codes E4M3, K/V codes E2M1; q6 (with
    fp4): Q codes E2M3.

    Qv, Kv, Vv: lists of float rows (original positions).  idx_list: the
    vertical positions of this KV head.  q/k/v codes and scales are per
    quantized row (already expanded: kscales[n] is the scale of row n's block).
    Returns a list of output rows (floats) and the weight rows.
    """
    D = len(Qv[0])
    alpha = 1.0 / math.sqrt(D)
    P = max(0, L - W)
    vl = set(idx_list)

    def cq(code):
        if q6:
            return float(e2m3_value_exact(code))
        return float(e4m3_value_exact(code)) if (fp8 or fp4) else int(code)

    def cv(code):
        if fp4:
            return float(e2m1_value_exact(code))
        return float(e4m3_value_exact(code)) if fp8 else int(code)
    qpos = [p for p in range(P) if p not in vl]          # quantized keys, ascending
    where = {p: n for n, p in enumerate(qpos)}
    out, weights = [], []
    for t in range(L):
        zs, vals, poss = [], [], []
        for p in range(t + 1):
            if bits != 16 and p in where and not (band and p >= t + 1 - W):
                n = where[p]
                dot = math.fsum(cq(qcodes[t][d]) * cv(kcodes[n][d]) for d in range(D))
                z = alpha * qscales[t // block] * kscales[n] * dot
                val = [vscales[n] * cv(vcodes[n][d]) for d in range(D)]
            else:
                z = alpha * math.fsum(Qv[t][d] * Kv[p][d] for d in range(D))
                val = list(Vv[p])
            zs.append(z)
            vals.append(val)
            poss.append(p)
        m = max(zs)
        ws = [math.exp(z - m) for z in zs]
        den = math.fsum(ws)
        row = [math.fsum(w * v[d] for w, v in zip(ws, vals)) / den for d in range(D)]
        wrow = [0.0] * L
        for p, w in zip(poss, ws):
            wrow[p] = w / den
        out.append(row)
        weights.append(wrow)
    return out, weights


def int_select(Qint, Kint, Hkv, W, k):
    """Selection on integer-valued inputs in exact int64 arithmetic:
    qsum = sum over group and tail, S = qsum . K, rank by (-S, p)."""
    B, Hq, L, D = Qint.shape
    g = Hq // Hkv
    t = min(W, L)
    P = max(0, L - W)
    out = np.zeros((B, Hkv, k), dtype=np.int64)
    for b in range(B):
        for j in range(Hkv):
            qs = Qint[b, j * g:(j + 1) * g, L - t:, :].astype(np.int64).sum(axis=(0, 1))
            S = Kint[b, j, :P, :].astype(np.int64) @ qs
            order = np.lexsort((np.arange(P), -S))
            out[b, j] = np.sort(order[:k])
    return out
