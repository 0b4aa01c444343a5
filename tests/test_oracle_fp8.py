"""Pins of the oracle's FP8 path: the E4M3 format (decode table, nearest-value
encoding), the per-block FP8 quantization of Algorithm 2 Stage 2 with
c_B = 448, and the hybrid attention computed from FP8 codes."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import brute
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen


def test_e4m3_table_matches_field_decoding():
    vals = orc.e4m3_values()
    for code in range(256):
        try:
            ref = brute.e4m3_value_exact(code)
        except ValueError:
            assert math.isnan(vals[code])
            continue
        assert Fraction(float(vals[code])) == ref
        assert math.copysign(1.0, vals[code]) == (-1.0 if code & 0x80 else 1.0)


def test_e4m3_named_values():
    v = orc.e4m3_values()
    assert v[0x7E] == 448.0 and v[0xFE] == -448.0          # largest finite (c_B)
    assert v[0x38] == 1.0
    assert v[0x08] == 2.0 ** -6                            # smallest normal
    assert v[0x01] == 2.0 ** -9                            # smallest subnormal
    assert v[0x07] == 7 * 2.0 ** -9                        # largest subnormal
    assert math.isnan(v[0x7F]) and math.isnan(v[0xFF])      # no infinities
    assert v[0x80] == 0.0 and math.copysign(1.0, v[0x80]) == -1.0
    finite = v[~np.isnan(v)]
    assert len(finite) == 254
    assert np.all(np.diff(v[:127]) > 0)                    # codes 0..126 ascend


def _probe_values(rng, n):
    mags = orc.e4m3_values()[:127]
    mids = 0.5 * (mags[:-1] + mags[1:])                    # exact ties between neighbours
    rand = rng.standard_normal(n) * np.exp2(rng.integers(-14, 10, n))
    edge = np.array([0.0, 448.0, 449.0, 464.0, 465.0, 1e4, 2.0 ** -10, 2.0 ** -11,
                     3 * 2.0 ** -11, 2.0 ** -9, 2.0 ** -6, 240.0, 256.0])
    vals = np.concatenate([mids, -mids, mags, -mags, rand, edge, -edge])
    return vals.astype(np.float32)


def test_e4m3_encode_matches_enumeration():
    y = _probe_values(np.random.default_rng(5), 400)
    codes = orc.e4m3_encode(y)
    for yi, ci in zip(y.tolist(), codes.tolist()):
        neg = math.copysign(1.0, yi) < 0
        assert ci == brute.e4m3_nearest(Fraction(yi), neg), (yi, ci)


def test_e4m3_encode_matches_torch_cast():
    """Library special case: torch's float32 -> float8_e4m3fn cast rounds to
    nearest-even; it agrees wherever it does not overflow (|y| < 464)."""
    y = _probe_values(np.random.default_rng(6), 2000)
    y = y[np.abs(y) < 464.0]
    ref = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(orc.e4m3_encode(y), ref)


def test_e4m3_roundtrip_every_finite_code():
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], np.uint8)
    vals = orc.e4m3_decode(codes).astype(np.float32)
    np.testing.assert_array_equal(orc.e4m3_encode(vals), codes)


def test_fp8_block_quant_matches_exact_rationals():
    rng = np.random.default_rng(448)
    for trial in range(40):
        n, D = int(rng.integers(1, 5)), int(rng.integers(1, 9))
        scale = float(10.0 ** rng.uniform(-20, 20))
        x = (rng.standard_normal((n, D)) * scale).astype(np.float32)
        x = gen.bf16_bits_to_f32(gen.f32_to_bf16_bits(x))
        codes, s = orc.quantize_rows_fp8(x, n)
        ref_codes, ref_s = brute.quant_block_fp8_exact(x.ravel())
        assert float(s[0]) == ref_s
        assert codes.ravel().tolist() == ref_codes


def test_fp8_block_quant_closed_forms():
    rng = np.random.default_rng(12)
    x = rng.standard_normal((64, 16)).astype(np.float32)
    codes, s = orc.quantize_rows_fp8(x, 64)
    i = np.unravel_index(np.argmax(np.abs(x)), x.shape)
    assert codes[i] == (0xFE if x[i] < 0 else 0x7E)                    # amax -> +-448
    # every code is the nearest E4M3 value: the error is at most half the gap
    # to the neighbouring magnitude
    mags = orc.e4m3_values()[:127]
    y = np.abs(x / s[0])
    dec = np.abs(orc.e4m3_decode(codes))
    k = np.searchsorted(mags, dec)                     # dec == mags[k]
    steps = np.diff(mags, prepend=0.0, append=np.inf)   # steps[i] = mags[i] - mags[i-1]
    gap = np.maximum(steps[k], steps[k + 1])           # to the neighbours below and above
    assert np.all(np.abs(y - dec) <= 0.5 * gap * (1 + 1e-6))
    zc, zs = orc.quantize_rows_fp8(np.zeros((3, 4), np.float32), 3)
    assert zs[0] == 0 and np.all(zc == 0)                              # all-zero block
    const = np.full((4, 8), -3.0, np.float32)
    cc, cs = orc.quantize_rows_fp8(const, 4)
    assert np.all(cc == 0xFE)                                          # constant -> -448


def test_fp8_needs_8_bit():
    d = gen.generate(1, 300, B=1, Hq=1, Hkv=1, L=64, D=8, W=8, plant=0.0)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 8, 0)
    with pytest.raises(ValueError):
        orc.quantize(d["Q"], d["K"], d["V"], idx, 8, 4, 16, fmt="fp8")


@pytest.mark.parametrize("L,D,W,ppm,block,Hq", [
    (40, 8, 6, 100000, 8, 1),
    (37, 4, 5, 200000, 5, 2),
])
def test_fp8_attention_brute_force_tiny(L, D, W, ppm, block, Hq):
    d = gen.generate(11, 301, B=1, Hq=Hq, Hkv=1, L=L, D=D, W=W, plant=0.1, outliers=(1,))
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, W, ppm)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, 8, block, fmt="fp8")
    O, Wt = orc.attention(d["Q"], d["K"], d["V"], W, 8, idx, qz, block, return_weights=True)
    P = max(0, L - W)
    vl = idx[0, 0].tolist()
    qpos = [p for p in range(P) if p not in set(vl)]
    for h in range(Hq):
        Qv = gen.bf16_bits_to_f32(d["Q"][0, h]).astype(np.float64).tolist()
        Kv = gen.bf16_bits_to_f32(d["K"][0, 0]).astype(np.float64).tolist()
        Vv = gen.bf16_bits_to_f32(d["V"][0, 0]).astype(np.float64).tolist()
        qc, qs = [], []
        for i in range(0, L, block):
            codes, s = brute.quant_block_fp8_exact(np.ravel(Qv[i:i + block]))
            qc += [codes[r * D:(r + 1) * D] for r in range(min(block, L - i))]
            qs.append(s)
        kc, ks, vc, vs = [], [], [], []
        for i in range(0, len(qpos), block):
            rows = qpos[i:i + block]
            codes, s = brute.quant_block_fp8_exact(np.ravel([Kv[p] for p in rows]))
            kc += [codes[r * D:(r + 1) * D] for r in range(len(rows))]
            ks += [s] * len(rows)
            codes, s = brute.quant_block_fp8_exact(np.ravel([Vv[p] for p in rows]))
            vc += [codes[r * D:(r + 1) * D] for r in range(len(rows))]
            vs += [s] * len(rows)
        out, wts = brute.attention_rows(Qv, Kv, Vv, L, W, 8, block, vl, qc, qs, kc, ks, vc, vs,
                                        fp8=True)
        np.testing.assert_allclose(O[h], np.array(out, np.float32), atol=1e-6, rtol=0)
        np.testing.assert_allclose(Wt[h], np.array(wts), atol=1e-12, rtol=0)


def test_fp8_hybrid_error_between_int8_and_exact():
    """Qualitative: with 3 mantissa bits the FP8 codes approximate the exact
    attention less well than int8 codes, and still far better than nothing
    (uniform weights)."""
    d = gen.generate(13, 302, B=1, Hq=2, Hkv=1, L=256, D=32, W=16, plant=0.02)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 16, 20000)
    exact = orc.attention(d["Q"], d["K"], d["V"], 16, 16, idx, None, 32)
    qi = orc.quantize(d["Q"], d["K"], d["V"], idx, 16, 8, 32)
    qf = orc.quantize(d["Q"], d["K"], d["V"], idx, 16, 8, 32, fmt="fp8")
    oi = orc.attention(d["Q"], d["K"], d["V"], 16, 8, idx, qi, 32)
    of = orc.attention(d["Q"], d["K"], d["V"], 16, 8, idx, qf, 32)
    ei = np.mean((oi - exact) ** 2)
    ef = np.mean((of - exact) ** 2)
    assert 0 < ei < ef < 1e-2 * np.mean(exact ** 2) + 1e-3
