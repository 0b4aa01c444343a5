"""CPU oracle for HyQuant hybrid-precision prefill attention.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow reference that the
HIP path is checked against.  Only the test suite, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it; the product
library never calls it and shares no code with it.

It follows the paper step by step:

* Algorithm 1 (App. A.1, Vertical Token Identification): window exclusion,
  tail-query proxy, GQA-native scoring, budget k and top-k.
* Algorithm 2 (App. A.2, HyQuant Prefill), Stage 1: the partition of the
  key positions into quantized / vertical-line / window sets (also the
  disjoint-partition equation of Section 4.1); Stage 2: per-tile symmetric
  quantization with scale max|x|/c_B.
* Eq. (prefill_hybrid) of Section 4.2: softmax over the concatenation of the
  dequantized-key logits and the full-precision logits, times the
  concatenation of the dequantized and full-precision values, here with a
  causal mask by original key position.  Attention is computed row-wise in
  float64 (not online), then rounded to float32.

Readings where the paper is silent or ambiguous (all fixed here, the HIP
path follows the same ones):

* the window is the last W keys [L-W, L); P = L - W is the prefix length;
* the vertical set is chosen per KV head, from the tail proxy summed over the
  g query heads of the group (the 1/t, 1/g means are dropped: they do not
  change the ranking);
* budget: k = 0 if the ratio is 0 or P = 0, else min(P, max(1, ceil(P*r)))
  with r given in parts per million and integer ceiling division;
* top-k ties go to the lowest position, -0 equals +0; the vertical index
  list is returned in ascending order;
* quantization blocks of ``block`` rows run over the compacted K_Q sequence
  (vertical-line rows removed) and over the original query rows; the scale
  is fl32(amax / c) and the code rint_half_even(fl32(x / s)) clamped to
  [-c, c]; an all-zero block has scale 0 and codes 0; c = 127 for 8-bit and
  7 for 4-bit; Q is always 8-bit when K/V are quantized;
* FP8 (Algorithm 2's second bit-width, c_B = 448): the format is OCP E4M3
  ("e4m3fn": no infinities, largest finite 448); the code of x is the E4M3
  value nearest to fl32(x / s), ties to the even code, saturating at +-448,
  the sign kept when the result is zero; Q, K_Q and V_Q all use it; codes
  are stored as their bit patterns (uint8);
* FP4 (the 4-bit floating-point format of the low-precision bulk path): OCP
  E2M1 (no infinities or NaN, largest finite 6) for K_Q and V_Q with
  c_B = 6, the code the E2M1 value nearest to fl32(x / s), ties to the even
  code, saturating at +-6, the sign kept when the result is zero; Q stays at
  8 bits in E4M3 (as with 4-bit integers, whose Q is int8); codes 0..15;
* FP4 with FP6 queries ("fp4q6"): K_Q and V_Q as for FP4; Q in OCP FP6
  E2M3 (no infinities or NaN, largest finite 7.5) with c_B = 7.5, the code
  the E2M3 value nearest to fl32(x / s), ties to the even code, saturating
  at +-7.5, the sign kept when the result is zero, one code per byte
  (bit 5 sign, bits 4..3 exponent, bits 2..0 mantissa), with the same
  per-64-row block scale as every other Q format; so that both operands of
  the quantized Q.K product are at most 6 bits wide;
* causality holds by original key position in every segment;
* bits = 16 disables quantization: every key takes the full-precision path.

Floating-point orders that the paper leaves open are pinned so that the
selection is reproducible bit for bit:

* tail proxy: for each query head r of the group, float32 sum of its tail
  rows in ascending row order starting from +0; then the g partial sums are
  added in head order;
* score: float32 products qsum[d]*K[p,d] (separate multiply, no fused
  multiply-add), then the upper half of the vector is folded onto the lower
  half repeatedly (128 -> 64 -> ... -> 1).
"""
from __future__ import annotations

import math

import numpy as np

C_INT8 = 127
C_INT4 = 7
C_FP8 = 448          # c_B for FP8 (Algorithm 2, Stage 2)
C_FP4 = 6            # c_B for FP4 E2M1: its largest finite value
C_FP6 = 7.5          # c_B for FP6 E2M3 queries: its largest finite value
FORMATS = ("int", "fp8", "fp4", "fp4q6")


# ---------------------------------------------------------------------------
# helpers
# ---------------------------------------------------------------------------

def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16/int16) -> float32, exact."""
    b = np.ascontiguousarray(bits).view(np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def code_bound(bits: int) -> int:
    """c_B of Algorithm 2, Stage 2 (127 for INT8); 7 for the 4-bit reading."""
    if bits == 8:
        return C_INT8
    if bits == 4:
        return C_INT4
    raise ValueError("no code bound for bits=%d" % bits)


def e4m3_values() -> np.ndarray:
    """Values of the 256 OCP FP8 E4M3 codes (float64): bit 7 sign, bits 6..3
    exponent with bias 7, bits 2..0 mantissa; exponent 0 is subnormal
    (m/8 * 2^-6); codes 0x7F and 0xFF are NaN; there are no infinities."""
    out = np.empty(256, dtype=np.float64)
    for code in range(256):
        sign = -1.0 if code & 0x80 else 1.0
        e = (code >> 3) & 0xF
        m = code & 0x7
        if e == 0xF and m == 0x7:
            out[code] = np.nan
        elif e == 0:
            out[code] = sign * (m / 8.0) * 2.0 ** -6
        else:
            out[code] = sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return out


_E4M3 = e4m3_values()


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """FP8 E4M3 bit patterns -> float64 values (exact)."""
    return _E4M3[np.asarray(codes).astype(np.uint8)]


def e4m3_encode(y: np.ndarray) -> np.ndarray:
    """float32 -> FP8 E4M3 bit patterns: the nearest finite E4M3 value, ties
    to the even code, |y| >= 448 saturating to +-448, the sign bit kept when
    the result is zero (-0 for negative inputs that round to 0)."""
    y = np.asarray(y, dtype=np.float32)
    mags = _E4M3[:127]                         # codes 0..126: 0 .. 448, ascending
    a = np.minimum(np.abs(y).astype(np.float64), 448.0)
    hi = np.clip(np.searchsorted(mags, a, side="left"), 1, 126)
    lo = hi - 1
    dlo = a - mags[lo]
    dhi = mags[hi] - a
    code = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(lo % 2 == 0, lo, hi)))
    code = code.astype(np.uint8)
    return np.where(np.signbit(y), code | np.uint8(0x80), code).astype(np.uint8)


def e2m1_values() -> np.ndarray:
    """Values of the 16 FP4 E2M1 codes (the OCP microscaling element format):
    bit 3 sign, bits 2..1 exponent with bias 1, bit 0 mantissa; exponent 0 is
    subnormal (m/2); no infinities, no NaN; largest finite value 6."""
    out = np.empty(16, dtype=np.float64)
    for code in range(16):
        sign = -1.0 if code & 0x8 else 1.0
        e = (code >> 1) & 0x3
        m = code & 0x1
        out[code] = sign * (m / 2.0 if e == 0 else (1.0 + m / 2.0) * 2.0 ** (e - 1))
    return out


_E2M1 = e2m1_values()


def e2m1_decode(codes: np.ndarray) -> np.ndarray:
    """FP4 E2M1 codes (0..15) -> float64 values (exact)."""
    return _E2M1[np.asarray(codes).astype(np.uint8) & 0xF]


def e2m1_encode(y: np.ndarray) -> np.ndarray:
    """float32 -> FP4 E2M1 codes (uint8, 0..15): the nearest of the eight
    magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6, ties to the even code, |y| beyond 6
    saturating to 6, the sign bit kept when the result is zero."""
    y = np.asarray(y, dtype=np.float32)
    mags = _E2M1[:8]                          # codes 0..7, ascending
    a = np.minimum(np.abs(y).astype(np.float64), 6.0)
    d = np.abs(a[..., None] - mags)           # distance to every magnitude
    best = d.min(axis=-1, keepdims=True)
    # among the nearest, the even code (two nearest codes are always adjacent)
    cand = np.where(d == best, np.arange(8), 99)
    even = np.where(cand % 2 == 0, cand, 99).min(axis=-1)
    code = np.where(even < 99, even, cand.min(axis=-1)).astype(np.uint8)
    return np.where(np.signbit(y), code | np.uint8(0x8), code).astype(np.uint8)


def e2m3_values() -> np.ndarray:
    """Values of the 64 FP6 E2M3 codes (the OCP microscaling element format):
    bit 5 sign, bits 4..3 exponent with bias 1, bits 2..0 mantissa; exponent
    0 is subnormal (m/8); no infinities, no NaN; largest finite value 7.5."""
    out = np.empty(64, dtype=np.float64)
    for code in range(64):
        sign = -1.0 if code & 0x20 else 1.0
        e = (code >> 3) & 0x3
        m = code & 0x7
        out[code] = sign * (m / 8.0 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 1))
    return out


_E2M3 = e2m3_values()


def e2m3_decode(codes: np.ndarray) -> np.ndarray:
    """FP6 E2M3 codes (0..63) -> float64 values (exact)."""
    return _E2M3[np.asarray(codes).astype(np.uint8) & 0x3F]


def e2m3_encode(y: np.ndarray) -> np.ndarray:
    """float32 -> FP6 E2M3 codes (uint8, 0..63): the nearest of the 32
    magnitudes 0 .. 7.5, ties to the even code, |y| beyond 7.5 saturating to
    7.5, the sign bit kept when the result is zero."""
    y = np.asarray(y, dtype=np.float32)
    mags = _E2M3[:32]                          # codes 0..31, ascending
    a = np.minimum(np.abs(y).astype(np.float64), C_FP6)
    hi = np.clip(np.searchsorted(mags, a, side="left"), 1, 31)
    lo = hi - 1
    dlo = a - mags[lo]
    dhi = mags[hi] - a
    code = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(lo % 2 == 0, lo, hi)))
    code = code.astype(np.uint8)
    return np.where(np.signbit(y), code | np.uint8(0x20), code).astype(np.uint8)


def q_code_values(codes: np.ndarray, fmt: str) -> np.ndarray:
    """The numbers the stored Q codes stand for (float64): E4M3 for FP8 and
    FP4 (which keeps the query at 8 bits), E2M3 for FP4 with FP6 queries,
    else integers."""
    if fmt in ("fp8", "fp4"):
        return e4m3_decode(codes)
    if fmt == "fp4q6":
        return e2m3_decode(codes)
    return np.asarray(codes).astype(np.float64)


def kv_code_values(codes: np.ndarray, fmt: str) -> np.ndarray:
    """The numbers the stored K/V codes stand for (float64)."""
    if fmt == "fp8":
        return e4m3_decode(codes)
    if fmt in ("fp4", "fp4q6"):
        return e2m1_decode(codes)
    return np.asarray(codes).astype(np.float64)


def sizes(L: int, W: int, budget_ppm: int, block: int = 64) -> dict:
    """Prefix length P, vertical budget k and block counts.

    P = max(0, L - W) (Algorithm 1, window exclusion); k = min(P, max(1,
    ceil(P * r))) (Algorithm 1, budget), r = budget_ppm / 1e6, and k = 0 when
    the budget is 0 or P = 0.  nQ = P - k keys are quantized.
    """
    if L < 1 or W < 0 or not (0 <= budget_ppm <= 1_000_000) or block < 1:
        raise ValueError("bad sizes arguments")
    P = max(0, L - W)
    if budget_ppm == 0 or P == 0:
        k = 0
    else:
        k = min(P, max(1, -(-(P * budget_ppm) // 1_000_000)))
    nQ = P - k
    return dict(P=P, k=k, nQ=nQ,
                n_qblk=-(-L // block),
                n_kvblk=-(-nQ // block))


# ---------------------------------------------------------------------------
# Algorithm 1: vertical token identification
# ---------------------------------------------------------------------------

def tail_proxy(Qf: np.ndarray, Hkv: int, W: int) -> np.ndarray:
    """Summed tail query per KV head: qsum[b, j, :] (float32).

    Algorithm 1, tail-query proxy with t = min(W, L_Q); GQA reshape of the
    query heads into (H_KV, g) with consecutive grouping.  Summed, not
    averaged (scale does not change the ranking).  Pinned order: per query
    head, ascending rows from +0; then heads in order.
    """
    B, Hq, L, D = Qf.shape
    g = Hq // Hkv
    t = min(W, L)
    Qg = Qf.reshape(B, Hkv, g, L, D)
    total = None
    for r in range(g):
        a = np.zeros((B, Hkv, D), dtype=np.float32)
        for i in range(L - t, L):
            a = a + Qg[:, :, r, i, :]
        total = a if total is None else total + a
    return total


def fold_sum(prod: np.ndarray) -> np.ndarray:
    """Sum over the last axis by repeatedly adding the upper half onto the
    lower half (the pinned reduction tree); the axis length must be a power
    of two."""
    v = prod
    n = v.shape[-1]
    if n & (n - 1):
        raise ValueError("head dim must be a power of two")
    while n > 1:
        h = n // 2
        v = v[..., :h] + v[..., h:n]
        n = h
    return v[..., 0]


def scores(qsum: np.ndarray, Kf: np.ndarray, P: int) -> np.ndarray:
    """S[b, j, p] = qsum[b, j] . K[b, j, p] for p in [0, P) (Algorithm 1,
    GQA-native einsum over the non-window prefix), float32, pinned tree."""
    prod = qsum[:, :, None, :] * Kf[:, :, :P, :]
    return fold_sum(prod)


def topk_ascending(S: np.ndarray, k: int) -> np.ndarray:
    """The k largest scores of the last axis (ties: lowest position first),
    returned as ascending positions (eq. vl_topk; Algorithm 1, TopK)."""
    S = S + np.float32(0.0)          # -0 -> +0
    out = np.empty(S.shape[:-1] + (k,), dtype=np.int32)
    for ix in np.ndindex(*S.shape[:-1]):
        order = np.argsort(-S[ix], kind="stable")   # stable: equal scores keep position order
        out[ix] = np.sort(order[:k]).astype(np.int32)
    return out


def select_vertical(Qb: np.ndarray, Kb: np.ndarray, Hkv: int, W: int, budget_ppm: int):
    """Algorithm 1 on bf16 inputs.  Returns (idx [B,Hkv,k] int32 ascending,
    S [B,Hkv,P] float32 or None when k = 0)."""
    B, Hq, L, D = Qb.shape
    sz = sizes(L, W, budget_ppm)
    P, k = sz["P"], sz["k"]
    if k == 0:
        return np.zeros((B, Hkv, 0), dtype=np.int32), None
    if min(W, L) < 1:
        raise ValueError("a vertical budget needs a window of at least one query")
    t = min(W, L)
    qsum = tail_proxy(bf16_to_f32(Qb[:, :, L - t:, :]), Hkv, W)   # only the tail rows are read
    S = scores(qsum, bf16_to_f32(Kb), P)
    return topk_ascending(S, k), S


def column_mass(Qb: np.ndarray, Kb: np.ndarray, Hkv: int, W: int) -> np.ndarray:
    """Eq. (vl_score): S[b, j, k] = sum over the considered queries of their
    attention probability on key k, for every key k in [0, L) (float64).

    The considered queries are the tail rows [L - t, L), t = min(W, L) (the
    rows Algorithm 1 summarizes) of the g query heads of KV head j; each
    probability is the plain causal softmax over keys <= the query's row of
    alpha * <q, k> with the bf16 inputs, alpha = 1/sqrt(D)."""
    B, Hq, L, D = Qb.shape
    g = Hq // Hkv
    t = min(W, L)
    rows = np.arange(L - t, L)
    alpha = 1.0 / math.sqrt(D)
    S = np.zeros((B, Hkv, L))
    for b in range(B):
        for j in range(Hkv):
            Kf = bf16_to_f32(Kb[b, j]).astype(np.float64)
            for r in range(g):
                q = bf16_to_f32(Qb[b, j * g + r][rows]).astype(np.float64)
                Z = alpha * (q @ Kf.T)
                Z = np.where(np.arange(L)[None, :] <= rows[:, None], Z, -np.inf)
                E = np.exp(Z - Z.max(axis=1, keepdims=True))
                S[b, j] += (E / E.sum(axis=1, keepdims=True)).sum(axis=0)
    return S


def select_vertical_colmass(Qb: np.ndarray, Kb: np.ndarray, Hkv: int, W: int, budget_ppm: int):
    """Eq. (vl_topk) on the exact column-mass score of eq. (vl_score): the k
    prefix keys [0, P) with the largest S (same budget k and tie rule as
    Algorithm 1).  Returns (idx [B,Hkv,k] int32 ascending, S [B,Hkv,P]
    float64 or None when k = 0)."""
    B, Hq, L, D = Qb.shape
    sz = sizes(L, W, budget_ppm)
    P, k = sz["P"], sz["k"]
    if k == 0:
        return np.zeros((B, Hkv, 0), dtype=np.int32), None
    if min(W, L) < 1:
        raise ValueError("a vertical budget needs a window of at least one query")
    S = column_mass(Qb, Kb, Hkv, W)[:, :, :P]
    out = np.empty((B, Hkv, k), dtype=np.int32)
    for ix in np.ndindex(B, Hkv):
        order = np.argsort(-S[ix], kind="stable")
        out[ix] = np.sort(order[:k]).astype(np.int32)
    return out, S


# ---------------------------------------------------------------------------
# Algorithm 2, Stages 1-2: partition and per-block quantization
# ---------------------------------------------------------------------------

def compaction(idx: np.ndarray, P: int) -> np.ndarray:
    """kq_pos[b, j, :] = [0, P) minus the vertical positions, ascending
    (Algorithm 2 Stage 1 partition; the K_Q index set of Algorithm 4)."""
    B, Hkv, k = idx.shape
    out = np.empty((B, Hkv, P - k), dtype=np.int32)
    for b in range(B):
        for j in range(Hkv):
            out[b, j] = np.setdiff1d(np.arange(P, dtype=np.int32), idx[b, j])
    return out


def quantize_rows(x: np.ndarray, block: int, c: int):
    """Per-block symmetric quantization of rows x [n, D] (float32).

    Algorithm 2 Stage 2: for each block of ``block`` consecutive rows, s =
    max|x| / c_B in float32, code = round(x / s) (half to even, float32
    division), clamped to [-c, c]; s = 0 gives codes 0.  Returns (codes int8
    [n, D], scales float32 [ceil(n/block)]).
    """
    n, D = x.shape
    nb = -(-n // block)
    padded = np.zeros((nb * block, D), dtype=np.float32)   # zero rows do not change max|x|
    padded[:n] = x
    blocks = padded.reshape(nb, block, D)
    amax = np.abs(blocks).max(axis=(1, 2))
    scales = (amax / np.float32(c)).astype(np.float32)      # float32 division per block
    safe = np.where(scales == 0, np.float32(1.0), scales)
    codes = np.clip(np.rint(blocks / safe[:, None, None]), -c, c)
    codes[scales == 0] = 0
    return codes.reshape(nb * block, D)[:n].astype(np.int8), scales


def quantize_rows_fp8(x: np.ndarray, block: int):
    """Per-block FP8 quantization of rows x [n, D] (float32): Algorithm 2
    Stage 2 with c_B = 448, s = fl32(max|x| / 448), code = E4M3(fl32(x / s));
    s = 0 gives codes 0.  Returns (codes uint8 [n, D], scales float32)."""
    n, D = x.shape
    nb = -(-n // block)
    padded = np.zeros((nb * block, D), dtype=np.float32)
    padded[:n] = x
    blocks = padded.reshape(nb, block, D)
    amax = np.abs(blocks).max(axis=(1, 2))
    scales = (amax / np.float32(C_FP8)).astype(np.float32)
    safe = np.where(scales == 0, np.float32(1.0), scales)
    codes = e4m3_encode((blocks / safe[:, None, None]).astype(np.float32))
    codes[scales == 0] = 0
    return codes.reshape(nb * block, D)[:n], scales


def quantize_rows_fp4(x: np.ndarray, block: int):
    """Per-block FP4 quantization of rows x [n, D] (float32): Algorithm 2
    Stage 2 with B = FP4 E2M1, c_B = 6, s = fl32(max|x| / 6), code =
    E2M1(fl32(x / s)); s = 0 gives codes 0.  Returns (codes uint8 [n, D] in
    0..15, scales float32)."""
    n, D = x.shape
    nb = -(-n // block)
    padded = np.zeros((nb * block, D), dtype=np.float32)
    padded[:n] = x
    blocks = padded.reshape(nb, block, D)
    amax = np.abs(blocks).max(axis=(1, 2))
    scales = (amax / np.float32(C_FP4)).astype(np.float32)
    safe = np.where(scales == 0, np.float32(1.0), scales)
    codes = e2m1_encode((blocks / safe[:, None, None]).astype(np.float32))
    codes[scales == 0] = 0
    return codes.reshape(nb * block, D)[:n], scales


def quantize_rows_fp6(x: np.ndarray, block: int):
    """Per-block FP6 quantization of rows x [n, D] (float32): Algorithm 2
    Stage 2 with B = FP6 E2M3, c_B = 7.5, s = fl32(max|x| / 7.5), code =
    E2M3(fl32(x / s)); s = 0 gives codes 0.  Returns (codes uint8 [n, D] in
    0..63, scales float32)."""
    n, D = x.shape
    nb = -(-n // block)
    padded = np.zeros((nb * block, D), dtype=np.float32)
    padded[:n] = x
    blocks = padded.reshape(nb, block, D)
    amax = np.abs(blocks).max(axis=(1, 2))
    scales = (amax / np.float32(C_FP6)).astype(np.float32)
    safe = np.where(scales == 0, np.float32(1.0), scales)
    codes = e2m3_encode((blocks / safe[:, None, None]).astype(np.float32))
    codes[scales == 0] = 0
    return codes.reshape(nb * block, D)[:n], scales


def quantize(Qb, Kb, Vb, idx, W: int, bits: int, block: int = 64, fmt: str = "int"):
    """Algorithm 2, Stages 1-2 on bf16 inputs.

    Returns a dict: kq_pos [B,Hkv,nQ]; q_codes [B,Hq,L,D], q_scale
    [B,Hq,n_qblk]; k_codes / v_codes [B,Hkv,nQ,D] (not packed), k_scale /
    v_scale [B,Hkv,n_kvblk].  ``fmt`` "int": int8 codes in [-c, c]; "fp8"
    (bits must be 8): E4M3 bit patterns (uint8) for Q, K and V; "fp4" (bits
    must be 4): E2M1 codes (uint8, 0..15) for K and V, E4M3 for Q; "fp4q6"
    (bits must be 4): E2M1 for K and V, E2M3 codes (uint8, 0..63) for Q.
    bits = 16 returns only kq_pos (nothing is quantized).
    """
    if fmt not in FORMATS or (fmt == "fp8" and bits != 8) or \
            (fmt in ("fp4", "fp4q6") and bits != 4):
        raise ValueError("fmt must be 'int', 'fp8' with bits = 8, or 'fp4' / 'fp4q6' with "
                         "bits = 4")
    B, Hq, L, D = Qb.shape
    Hkv = Kb.shape[1]
    P = max(0, L - W)
    kq_pos = compaction(idx, P)
    out = dict(kq_pos=kq_pos)
    if bits == 16:
        return out
    nQ = kq_pos.shape[2]
    n_qblk = -(-L // block)
    n_kvblk = -(-nQ // block)
    if fmt == "fp8":
        def qrows(x, c):
            return quantize_rows_fp8(x, block)
        q_rows = qrows
        ctype = np.uint8
    elif fmt in ("fp4", "fp4q6"):
        def qrows(x, c):
            return quantize_rows_fp4(x, block)

        def q_rows(x, c):
            return quantize_rows_fp8(x, block) if fmt == "fp4" else quantize_rows_fp6(x, block)
        ctype = np.uint8
    else:
        def qrows(x, c):
            return quantize_rows(x, block, c)
        q_rows = qrows
        ctype = np.int8
    c = code_bound(bits)
    q_codes = np.zeros((B, Hq, L, D), ctype)
    q_scale = np.zeros((B, Hq, n_qblk), np.float32)
    for b in range(B):
        for h in range(Hq):
            q_codes[b, h], q_scale[b, h] = q_rows(bf16_to_f32(Qb[b, h]), C_INT8)
    k_codes = np.zeros((B, Hkv, nQ, D), ctype)
    v_codes = np.zeros((B, Hkv, nQ, D), ctype)
    k_scale = np.zeros((B, Hkv, n_kvblk), np.float32)
    v_scale = np.zeros((B, Hkv, n_kvblk), np.float32)
    for b in range(B):
        for j in range(Hkv):
            rows = kq_pos[b, j]
            k_codes[b, j], k_scale[b, j] = qrows(bf16_to_f32(Kb[b, j][rows]), c)
            v_codes[b, j], v_scale[b, j] = qrows(bf16_to_f32(Vb[b, j][rows]), c)
    out.update(q_codes=q_codes, q_scale=q_scale, k_codes=k_codes, k_scale=k_scale,
               v_codes=v_codes, v_scale=v_scale, fmt=fmt)
    return out


# ---------------------------------------------------------------------------
# Eq. (prefill_hybrid): hybrid-precision causal attention
# ---------------------------------------------------------------------------

WINDOW_MODES = ("fixed", "band")


def _head_operands(Qb, Kb, Vb, b, h, Hkv, W, bits, block, idx, qz, window_mode="fixed"):
    """Logit ingredients of one (batch, query head): for every key, the rows
    that see it (lo <= t <= hi, original positions), and the pieces of its
    logit and value.

    window_mode "fixed": the full-precision window is the last W keys [P, L)
    (Algorithms 1, 2, 4); a key is seen by every row t >= its position.
    window_mode "band": the per-query window of eq. (win_def) with t0 = t + 1,
    i.e. row t sees keys [t + 1 - W, t] in full precision; other keys of the
    non-window prefix only quantized (position <= t - W); vertical lines in
    full precision from their position on (eq. pre_def: the prefix is the
    complement of the window of the current query).
    """
    B, Hq, L, D = Qb.shape
    g = Hq // Hkv
    j = h // g
    P = max(0, L - W)
    big = np.iinfo(np.int64).max
    if bits == 16:
        fp_pos = np.arange(L)
        fp_hi = np.full(L, big)
    elif window_mode == "fixed":
        fp_pos = np.concatenate([idx[b, j].astype(np.int64), np.arange(P, L)])
        fp_hi = np.full(len(fp_pos), big)
    else:
        vlp = idx[b, j].astype(np.int64)
        rest = np.setdiff1d(np.arange(L), vlp)            # every non-vertical key, ascending
        fp_pos = np.concatenate([vlp, rest])
        fp_hi = np.concatenate([np.full(len(vlp), big), rest + W - 1])
    ops = dict(
        fp_pos=fp_pos,
        fp_lo=fp_pos,
        fp_hi=fp_hi,
        Q=bf16_to_f32(Qb[b, h]).astype(np.float64),
        Kfp=bf16_to_f32(Kb[b, j][fp_pos]).astype(np.float64),
        Vfp=bf16_to_f32(Vb[b, j][fp_pos]).astype(np.float64),
    )
    if bits != 16:
        nQ = qz["kq_pos"].shape[2]
        blk = np.arange(nQ) // block
        fmt = qz.get("fmt", "int")
        q_pos = qz["kq_pos"][b, j].astype(np.int64)
        ops.update(
            q_pos=q_pos,
            q_lo=q_pos + (W if window_mode == "band" else 0),
            qcode=q_code_values(qz["q_codes"][b, h], fmt),
            qscale=qz["q_scale"][b, h].astype(np.float64),
            kcode=kv_code_values(qz["k_codes"][b, j], fmt),
            kscale=qz["k_scale"][b, j][blk].astype(np.float64),
            vhat=qz["v_scale"][b, j][blk].astype(np.float64)[:, None] * kv_code_values(qz["v_codes"][b, j], fmt),
        )
    return ops


def _rows_logits(ops, rows, D, bits, block):
    """Concatenated logits [len(rows), nkeys], values, key positions and the
    first / last row that sees each key."""
    alpha = 1.0 / math.sqrt(D)
    Zfp = alpha * (ops["Q"][rows] @ ops["Kfp"].T)
    if bits == 16:
        return Zfp, ops["Vfp"], ops["fp_pos"], ops["fp_lo"], ops["fp_hi"]
    # Quantized keys: alpha * s_Q * s_K * <q_code, k_code> (Algorithm 2, Segment A).
    Zq = alpha * (ops["qcode"][rows] @ ops["kcode"].T) \
        * ops["qscale"][rows // block][:, None] * ops["kscale"][None, :]
    Z = np.concatenate([Zq, Zfp], axis=1)
    Vall = np.concatenate([ops["vhat"], ops["Vfp"]], axis=0)
    pos = np.concatenate([ops["q_pos"], ops["fp_pos"]])
    lo = np.concatenate([ops["q_lo"], ops["fp_lo"]])
    hi = np.concatenate([np.full(len(ops["q_pos"]), np.iinfo(np.int64).max), ops["fp_hi"]])
    return Z, Vall, pos, lo, hi


def attention(Qb, Kb, Vb, W: int, bits: int, idx, qz=None, block: int = 64,
              heads=None, rows=None, return_weights: bool = False, chunk: int = 1024,
              window_mode: str = "fixed"):
    """Causal hybrid attention output in float32.

    ``heads``: list of (b, h) to evaluate (default: all); ``rows``: query rows
    (default: all), shared by every listed head.  ``window_mode``: "fixed"
    or "band" (see _head_operands).  Returns O [len(heads), len(rows), D]
    float32 (and, if ``return_weights``, the float64 weight matrices over
    original key positions [len(heads), len(rows), L]; in band mode a
    position's quantized and full-precision weights are added).
    """
    if window_mode not in WINDOW_MODES:
        raise ValueError(f"window_mode must be one of {WINDOW_MODES}")
    B, Hq, L, D = Qb.shape
    Hkv = Kb.shape[1]
    if heads is None:
        heads = [(b, h) for b in range(B) for h in range(Hq)]
    rows = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    O = np.zeros((len(heads), len(rows), D), dtype=np.float32)
    Wfull = np.zeros((len(heads), len(rows), L)) if return_weights else None
    for hi_, (b, h) in enumerate(heads):
        ops = _head_operands(Qb, Kb, Vb, b, h, Hkv, W, bits, block, idx, qz, window_mode)
        nkeys = len(ops["fp_pos"]) + (len(ops["q_pos"]) if bits != 16 else 0)
        step = max(1, min(chunk, (1 << 25) // max(1, nkeys)))
        for c0 in range(0, len(rows), step):
            r = rows[c0:c0 + step]
            Z, Vall, pos, lo, hi = _rows_logits(ops, r, D, bits, block)
            seen = (lo[None, :] <= r[:, None]) & (r[:, None] <= hi[None, :])
            Z = np.where(seen, Z, -np.inf)     # causal (and band), original positions
            m = Z.max(axis=1, keepdims=True)
            E = np.exp(Z - m)
            den = E.sum(axis=1, keepdims=True)
            O[hi_, c0:c0 + len(r)] = ((E @ Vall) / den).astype(np.float32)
            if return_weights:
                Wr = np.zeros((len(r), L))
                for kk in range(len(pos)):
                    Wr[:, pos[kk]] += E[:, kk] / den[:, 0]
                Wfull[hi_, c0:c0 + len(r)] = Wr
    return (O, Wfull) if return_weights else O


def attention_final_chunk(Qb, Kb, Vb, W: int, bits: int, idx, qz, block: int = 64,
                          tile: int = 64, heads=None):
    """Algorithm 2, Stage 3 taken literally for the final query chunk, the
    rows [L - W, L) (at most W rows): segment A (every quantized key) and
    segment B (every vertical-line key) without a mask, segment C (the window
    [L - W, L)) with the per-row causal mask; each segment scanned in tiles
    of ``tile`` keys with the online-softmax update FlashOS (running max m,
    sum l, accumulator), float64.  Returns O [len(heads), W', D] float32,
    W' = min(W, L)."""
    B, Hq, L, D = Qb.shape
    Hkv = Kb.shape[1]
    g = Hq // Hkv
    P = max(0, L - W)
    rows = np.arange(P, L)
    alpha = 1.0 / math.sqrt(D)
    if heads is None:
        heads = [(b, h) for b in range(B) for h in range(Hq)]
    O = np.zeros((len(heads), len(rows), D), dtype=np.float32)
    for hi_, (b, h) in enumerate(heads):
        j = h // g
        q = bf16_to_f32(Qb[b, h][rows]).astype(np.float64)
        Kf = bf16_to_f32(Kb[b, j]).astype(np.float64)
        Vf = bf16_to_f32(Vb[b, j]).astype(np.float64)
        m = np.full(len(rows), -np.inf)
        l = np.zeros(len(rows))
        acc = np.zeros((len(rows), D))

        def flash_os(z, v):
            nonlocal m, l, acc
            mn = np.maximum(m, z.max(axis=1))
            safe = np.where(np.isfinite(mn), mn, 0.0)
            corr = np.where(np.isfinite(m), np.exp(m - safe), 0.0)
            p = np.exp(z - safe[:, None])
            l = l * corr + p.sum(axis=1)
            acc = acc * corr[:, None] + p @ v
            m = mn

        if bits != 16:
            fmt = qz.get("fmt", "int")
            nQ = qz["kq_pos"].shape[2]
            qcode = q_code_values(qz["q_codes"][b, h][rows], fmt)
            qs = qz["q_scale"][b, h][rows // block].astype(np.float64)
            kcode = kv_code_values(qz["k_codes"][b, j], fmt)
            vcode = kv_code_values(qz["v_codes"][b, j], fmt)
            for t0 in range(0, nQ, tile):                  # segment A, no mask
                n = np.arange(t0, min(nQ, t0 + tile))
                ks = qz["k_scale"][b, j][n // block].astype(np.float64)
                vs = qz["v_scale"][b, j][n // block].astype(np.float64)
                z = alpha * (qcode @ kcode[n].T) * qs[:, None] * ks[None, :]
                flash_os(z, vs[:, None] * vcode[n])
            vlp = idx[b, j].astype(np.int64)
            for t0 in range(0, len(vlp), tile):            # segment B, no mask
                pp = vlp[t0:t0 + tile]
                flash_os(alpha * (q @ Kf[pp].T), Vf[pp])
        win = np.arange(P, L) if bits != 16 else np.arange(0, L)
        for t0 in range(0, len(win), tile):               # segment C, causal
            pp = win[t0:t0 + tile]
            z = alpha * (q @ Kf[pp].T)
            z = np.where(pp[None, :] <= rows[:, None], z, -np.inf)
            flash_os(z, Vf[pp])
        O[hi_] = (acc / l[:, None]).astype(np.float32)
    return O


def prefill(Qb, Kb, Vb, Hkv: int, W: int, budget_ppm: int, bits: int, block: int = 64,
            heads=None, rows=None, fmt: str = "int", window_mode: str = "fixed"):
    """The whole path of Algorithm 2: selection, quantization, attention."""
    idx, _ = select_vertical(Qb, Kb, Hkv, W, budget_ppm)
    qz = quantize(Qb, Kb, Vb, idx, W, bits, block, fmt)
    O = attention(Qb, Kb, Vb, W, bits, idx, qz, block, heads=heads, rows=rows,
                  window_mode=window_mode)
    return dict(idx=idx, O=O, **qz)


# ---------------------------------------------------------------------------
# Decode: Algorithm 4 (Freeze) and Algorithm 3 (HyQuant Decode)
# ---------------------------------------------------------------------------
#
# Readings (the paper leaves the staging policy open):
# * Freeze reuses the prefill steps exactly: Algorithm 1 on the prefill's
#   tail queries, the partition, and the per-block K/V quantization over the
#   compacted K_Q order; it keeps copies of the vertical-line rows and of the
#   last W rows (the window) and drops the full-precision cache.
# * The staging buffer holds up to Ws = 64 new tokens in full precision.
#   When a new token arrives and the staging buffer is full, it is merged
#   first: the Ws oldest window tokens are quantized as one new block of the
#   quantized prefix (the same formula, c_B and format), and the staging
#   tokens take their place in the window, which stays exactly W tokens.
#   Requires W >= Ws, and a prefill of N >= W tokens (so that the window is
#   full from the start).
# * The decode query is used in full precision (bf16 values); quantized keys
#   and values enter through their dequantized values s * code.  Every cached
#   key precedes the query: there is no mask.

DECODE_WS = 64


def freeze(Qb, Kb, Vb, Hkv: int, W: int, budget_ppm: int, bits: int, block: int = 64,
           fmt: str = "int", selector: str = "proxy", staging: int = DECODE_WS):
    """Algorithm 4 on a prefill of N tokens (bf16 inputs).  Returns the hybrid
    cache as a dict of numpy arrays (per (b, j) lists where sizes can grow):
    quantized prefix (kq_pos, k/v codes and scales per block), vertical-line
    rows, window rows, an empty staging buffer of capacity ``staging`` (W_s,
    a multiple of the block)."""
    if bits == 16:
        raise ValueError("freeze needs a quantized format (bits 8 or 4)")
    if fmt == "fp4q6":
        raise ValueError("decode keeps its queries in bf16: use fmt 'fp4' (the query "
                         "format of 'fp4q6' applies to the prefill only)")
    B, Hq, N, D = Qb.shape
    if staging < block or staging % block:
        raise ValueError("the staging capacity is a positive multiple of the block")
    if W < staging or N < W:
        raise ValueError("decode needs W >= Ws (merges move Ws window tokens) and N >= W")
    if selector == "colmass":
        idx, _ = select_vertical_colmass(Qb, Kb, Hkv, W, budget_ppm)
    else:
        idx, _ = select_vertical(Qb, Kb, Hkv, W, budget_ppm)
    qz = quantize(Qb, Kb, Vb, idx, W, bits, block, fmt)
    P = max(0, N - W)
    nq = qz["kq_pos"].shape[2]
    nb = -(-nq // block)
    cache = dict(B=B, Hq=Hq, Hkv=Hkv, D=D, W=W, bits=bits, fmt=fmt, block=block, t=N, idx=idx,
                 Ws=staging)
    kc, vc, ks, vs, pos = [], [], [], [], []
    for b in range(B):
        for j in range(Hkv):
            # blocks as lists: codes [n, D] (unpacked), positions; the last Freeze
            # block may be ragged (nq not a multiple of the block)
            kc.append([qz["k_codes"][b, j, i * block:(i + 1) * block] for i in range(nb)])
            vc.append([qz["v_codes"][b, j, i * block:(i + 1) * block] for i in range(nb)])
            ks.append(list(qz["k_scale"][b, j]))
            vs.append(list(qz["v_scale"][b, j]))
            pos.append([qz["kq_pos"][b, j, i * block:(i + 1) * block] for i in range(nb)])
    cache.update(k_blocks=kc, v_blocks=vc, k_scales=ks, v_scales=vs, q_pos=pos)
    cache["vl_k"] = np.stack([Kb[b, j][idx[b, j]] for b in range(B) for j in range(Hkv)])
    cache["vl_v"] = np.stack([Vb[b, j][idx[b, j]] for b in range(B) for j in range(Hkv)])
    cache["vl_pos"] = idx.reshape(B * Hkv, -1)
    # window as a list of rows per (b, j), oldest first
    cache["win_k"] = [list(Kb[b, j][P:N]) for b in range(B) for j in range(Hkv)]
    cache["win_v"] = [list(Vb[b, j][P:N]) for b in range(B) for j in range(Hkv)]
    cache["win_pos"] = [list(range(P, N)) for _ in range(B * Hkv)]
    cache["st_k"] = [[] for _ in range(B * Hkv)]
    cache["st_v"] = [[] for _ in range(B * Hkv)]
    cache["st_pos"] = [[] for _ in range(B * Hkv)]
    return cache


def _quantize_block(rows_f32: np.ndarray, cache):
    if cache["fmt"] == "fp8":
        return quantize_rows_fp8(rows_f32, rows_f32.shape[0])
    if cache["fmt"] == "fp4":
        return quantize_rows_fp4(rows_f32, rows_f32.shape[0])
    return quantize_rows(rows_f32, rows_f32.shape[0], code_bound(cache["bits"]))


def decode_merge(cache):
    """Staging full: quantize the Ws oldest window tokens into Ws / block new
    blocks of the quantized prefix (oldest first, each with its own scale,
    as Freeze quantizes); the staging tokens join the window."""
    Ws, G = cache["Ws"], cache["block"]
    for bj in range(cache["B"] * cache["Hkv"]):
        if cache["W"] < Ws or len(cache["st_k"][bj]) != Ws:
            raise ValueError("merge needs W >= Ws and a full staging buffer")
        for i in range(0, Ws, G):
            ek = bf16_to_f32(np.stack(cache["win_k"][bj][i:i + G]))
            ev = bf16_to_f32(np.stack(cache["win_v"][bj][i:i + G]))
            kcode, ksc = _quantize_block(ek, cache)
            vcode, vsc = _quantize_block(ev, cache)
            cache["k_blocks"][bj].append(kcode)
            cache["v_blocks"][bj].append(vcode)
            cache["k_scales"][bj].append(ksc[0])
            cache["v_scales"][bj].append(vsc[0])
            cache["q_pos"][bj].append(np.array(cache["win_pos"][bj][i:i + G], np.int32))
        for name in ("k", "v", "pos"):
            w, st = cache["win_" + name], cache["st_" + name]
            w[bj] = w[bj][Ws:] + st[bj]
            st[bj] = []


def decode_append(cache, k_new, v_new):
    """One new token's key and value rows (bf16 bits [B, Hkv, D]) enter the
    staging buffer (merging it first if it is full)."""
    if len(cache["st_k"][0]) == cache["Ws"]:
        decode_merge(cache)
    t = cache["t"]
    for b in range(cache["B"]):
        for j in range(cache["Hkv"]):
            bj = b * cache["Hkv"] + j
            cache["st_k"][bj].append(np.asarray(k_new[b, j]))
            cache["st_v"][bj].append(np.asarray(v_new[b, j]))
            cache["st_pos"][bj].append(t)
    cache["t"] = t + 1


def decode_keys(cache, bj):
    """Every cached key of KV head bj with its value and original position:
    (K [n, D] float64, V [n, D] float64, pos [n]); quantized keys dequantized
    as scale * value(code)."""
    fmt = cache["fmt"]
    Ks, Vs, Ps = [], [], []
    for kc, vc, ksc, vsc, pos in zip(cache["k_blocks"][bj], cache["v_blocks"][bj],
                                     cache["k_scales"][bj], cache["v_scales"][bj],
                                     cache["q_pos"][bj]):
        n = len(pos)
        Ks.append(np.float64(ksc) * kv_code_values(kc[:n], fmt))
        Vs.append(np.float64(vsc) * kv_code_values(vc[:n], fmt))
        Ps.append(np.asarray(pos, np.int64))
    for kk, vv, pp in ((cache["vl_k"][bj], cache["vl_v"][bj], cache["vl_pos"][bj]),
                       (cache["win_k"][bj], cache["win_v"][bj], cache["win_pos"][bj]),
                       (cache["st_k"][bj], cache["st_v"][bj], cache["st_pos"][bj])):
        if len(pp):
            Ks.append(bf16_to_f32(np.stack(kk)).astype(np.float64))
            Vs.append(bf16_to_f32(np.stack(vv)).astype(np.float64))
            Ps.append(np.asarray(pp, np.int64))
    return np.concatenate(Ks), np.concatenate(Vs), np.concatenate(Ps)


def decode_attention(q_bits, cache):
    """Algorithm 3 for one decode query per (batch, query head): softmax of
    alpha * q . k over every cached key (float64, one plain row-wise softmax),
    times the values; returns O [B, Hq, D] float32."""
    B, Hq, Hkv, D = cache["B"], cache["Hq"], cache["Hkv"], cache["D"]
    g = Hq // Hkv
    alpha = 1.0 / math.sqrt(D)
    q = bf16_to_f32(q_bits).astype(np.float64)
    O = np.zeros((B, Hq, D), np.float32)
    for b in range(B):
        for j in range(Hkv):
            Kall, Vall, _ = decode_keys(cache, b * Hkv + j)
            for r in range(g):
                h = j * g + r
                z = alpha * (Kall @ q[b, h])
                e = np.exp(z - z.max())
                O[b, h] = ((e @ Vall) / e.sum()).astype(np.float32)
    return O
