"""Pins of the oracle's window readings: the per-query window of eq. (win_def)
/ eq. (pre_def) ("band" mode: row t sees keys t+1-W .. t in full precision),
and Algorithm 2's Stage 3 taken literally for the final query chunk (segments
A and B without a mask, segment C causal), scanned tile by tile with the
online-softmax update."""
import math

import numpy as np
import pytest

import brute
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen


def sdpa_causal_rows(Qb, Kb, Vb, b, h, Hkv, rows):
    g = Qb.shape[1] // Hkv
    q = gen.bf16_bits_to_f32(Qb[b, h]).astype(np.float64)
    k = gen.bf16_bits_to_f32(Kb[b, h // g]).astype(np.float64)
    v = gen.bf16_bits_to_f32(Vb[b, h // g]).astype(np.float64)
    out = []
    for t in rows:
        z = (k[:t + 1] @ q[t]) / math.sqrt(q.shape[1])
        e = np.exp(z - z.max())
        out.append((e @ v[:t + 1]) / e.sum())
    return np.array(out)


def _setup(seed, L, D, W, ppm, bits, Hq=2, Hkv=1, fmt="int", block=64):
    d = gen.generate(seed, 700 + seed, B=1, Hq=Hq, Hkv=Hkv, L=L, D=D, W=max(W, 1), plant=0.05)
    idx, _ = orc.select_vertical(d["Q"], d["K"], Hkv, W, ppm)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, bits, block, fmt) if bits != 16 else None
    return d, idx, qz


def test_band_rows_before_W_are_exact_attention():
    """Row t < W sees all of [0, t] in full precision, although quantized keys
    exist (they are only visible to rows t >= position + W)."""
    L, D, W = 200, 16, 48
    d, idx, qz = _setup(1, L, D, W, 30000, 8)
    assert qz["kq_pos"].shape[2] > 0
    rows = np.arange(0, W)
    O = orc.attention(d["Q"], d["K"], d["V"], W, 8, idx, qz, heads=[(0, 1)], rows=rows,
                      window_mode="band")[0]
    ref = sdpa_causal_rows(d["Q"], d["K"], d["V"], 0, 1, 1, rows)
    np.testing.assert_allclose(O, ref, atol=2e-7, rtol=0)
    # ... while the fixed reading quantizes the early prefix for the same rows
    Of = orc.attention(d["Q"], d["K"], d["V"], W, 8, idx, qz, heads=[(0, 1)], rows=rows)[0]
    assert np.abs(Of - ref).max() > 1e-5


def test_band_width_zero_is_uniform_quantization_of_fixed_reading():
    L, D = 150, 8
    d, idx, qz = _setup(2, L, D, 0, 0, 8)
    Ob = orc.attention(d["Q"], d["K"], d["V"], 0, 8, idx, qz, window_mode="band")
    Of = orc.attention(d["Q"], d["K"], d["V"], 0, 8, idx, qz)
    np.testing.assert_array_equal(Ob, Of)


@pytest.mark.parametrize("bits,fmt", [(8, "int"), (4, "int"), (8, "fp8")])
def test_band_last_row_equals_fixed_reading(bits, fmt):
    """For the last row t = L-1 the band [L-W, L-1] is the fixed window and
    every quantized key is older than it: both readings agree."""
    L, D, W = 260, 16, 40
    d, idx, qz = _setup(3, L, D, W, 40000, bits, fmt=fmt)
    rows = np.array([L - 1])
    Ob = orc.attention(d["Q"], d["K"], d["V"], W, bits, idx, qz, rows=rows, window_mode="band")
    Of = orc.attention(d["Q"], d["K"], d["V"], W, bits, idx, qz, rows=rows)
    np.testing.assert_allclose(Ob, Of, atol=1e-7, rtol=0)


@pytest.mark.parametrize("L,D,W,ppm,bits,block,fp8", [
    (24, 4, 5, 150000, 8, 4, False),
    (20, 8, 3, 100000, 4, 2, False),
    (22, 4, 6, 200000, 8, 3, True),
])
def test_band_brute_force_tiny(L, D, W, ppm, bits, block, fp8):
    fmt = "fp8" if fp8 else "int"
    d = gen.generate(9, 710, B=1, Hq=1, Hkv=1, L=L, D=D, W=W, plant=0.1, outliers=(1,))
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, W, ppm)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, bits, block, fmt)
    O, Wt = orc.attention(d["Q"], d["K"], d["V"], W, bits, idx, qz, block, return_weights=True,
                          window_mode="band")
    P = max(0, L - W)
    vl = idx[0, 0].tolist()
    qpos = [p for p in range(P) if p not in set(vl)]
    Qv = gen.bf16_bits_to_f32(d["Q"][0, 0]).astype(np.float64).tolist()
    Kv = gen.bf16_bits_to_f32(d["K"][0, 0]).astype(np.float64).tolist()
    Vv = gen.bf16_bits_to_f32(d["V"][0, 0]).astype(np.float64).tolist()
    quant = brute.quant_block_fp8_exact if fp8 else (
        lambda x: brute.quant_block_exact(x, orc.code_bound(bits)))
    qc, qs = [], []
    for i in range(0, L, block):
        codes, s = brute.quant_block_fp8_exact(np.ravel(Qv[i:i + block])) if fp8 else \
            brute.quant_block_exact(np.ravel(Qv[i:i + block]), 127)
        qc += [codes[r * D:(r + 1) * D] for r in range(min(block, L - i))]
        qs.append(s)
    kc, ks, vc, vs = [], [], [], []
    for i in range(0, len(qpos), block):
        rws = qpos[i:i + block]
        codes, s = quant(np.ravel([Kv[p] for p in rws]))
        kc += [codes[r * D:(r + 1) * D] for r in range(len(rws))]
        ks += [s] * len(rws)
        codes, s = quant(np.ravel([Vv[p] for p in rws]))
        vc += [codes[r * D:(r + 1) * D] for r in range(len(rws))]
        vs += [s] * len(rws)
    out, wts = brute.attention_rows(Qv, Kv, Vv, L, W, bits, block, vl, qc, qs, kc, ks, vc, vs,
                                    fp8=fp8, band=True)
    np.testing.assert_allclose(O[0], np.array(out, np.float32), atol=1e-6, rtol=0)
    np.testing.assert_allclose(Wt[0], np.array(wts), atol=1e-12, rtol=0)


def test_band_rows_sum_to_one_and_causal():
    L, D, W = 180, 8, 32
    d, idx, qz = _setup(4, L, D, W, 50000, 4)
    _, Wt = orc.attention(d["Q"], d["K"], d["V"], W, 4, idx, qz, return_weights=True,
                          window_mode="band")
    np.testing.assert_allclose(Wt.sum(-1), 1.0, atol=1e-12)
    assert np.all(np.triu(Wt[0, 0], 1) == 0) and np.all(np.triu(Wt[1, 0], 1) == 0)


@pytest.mark.parametrize("L,D,W,ppm,bits,fmt,tile", [
    (300, 16, 64, 30000, 8, "int", 64),
    (257, 16, 40, 50000, 4, "int", 16),
    (200, 8, 50, 20000, 8, "fp8", 7),
    (130, 8, 30, 0, 8, "int", 64),          # no vertical lines
    (90, 8, 20, 10000, 16, "int", 64),      # nothing quantized: C covers every key
])
def test_literal_final_chunk_equals_causal_reading(L, D, W, ppm, bits, fmt, tile):
    """For the final chunk of W rows, Algorithm 2's literal Stage 3 (A and B
    unmasked, C causal, tile-by-tile online softmax) equals the
    whole-sequence causal definition: every quantized and vertical key
    precedes the chunk."""
    d, idx, qz = _setup(5, L, D, W, ppm, bits, Hq=4, Hkv=2, fmt=fmt)
    Oc = orc.attention_final_chunk(d["Q"], d["K"], d["V"], W, bits, idx, qz, tile=tile)
    rows = np.arange(L - W, L)
    Od = orc.attention(d["Q"], d["K"], d["V"], W, bits, idx, qz, rows=rows)
    np.testing.assert_allclose(Oc, Od, atol=2e-7, rtol=0)


def test_literal_form_needs_causality_before_the_final_chunk():
    """The same unmasked segments A/B applied to a row before the final chunk
    would let it attend to later keys: the literal form is only the final
    chunk's (hence the causal mask in every segment for a whole prefill)."""
    L, D, W = 200, 8, 40
    d, idx, qz = _setup(6, L, D, W, 30000, 8)
    P = L - W
    t = P // 2
    # a later quantized key is visible in the literal form: its position exceeds t
    assert np.any(qz["kq_pos"][0, 0] > t) and np.any(qz["kq_pos"][0, 0] < P)
