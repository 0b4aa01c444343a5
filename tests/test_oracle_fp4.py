"""Pins of the oracle's FP4 format (OCP E2M1 K/V codes with c_B = 6, E4M3
queries): the value table, the encoding against exact-rational enumeration,
block quantization against exact rationals and closed forms, and attention
against a scalar-loop brute force with its own quantization."""
from fractions import Fraction

import numpy as np
import pytest

import brute
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen


def test_e2m1_named_values():
    """The OCP microscaling FP4 element values: 0, 0.5, 1, 1.5, 2, 3, 4, 6 and
    their negatives (code 8 is -0)."""
    v = orc.e2m1_values()
    assert v[:8].tolist() == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
    assert v[8:].tolist() == [-0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0]
    assert np.signbit(v[8]) and not np.signbit(v[0])


def test_e2m1_table_matches_field_decoding():
    for code in range(16):
        assert Fraction(float(orc.e2m1_values()[code])) == brute.e2m1_value_exact(code)


def _probe_values():
    """Every value, every midpoint and their float32 neighbours (two ulps each
    way), plus saturating and tiny inputs."""
    mags = [0, 0.5, 1, 1.5, 2, 3, 4, 6]
    pts = set()
    for a, b in zip(mags, mags[1:]):
        for x in (a, b, (a + b) / 2):
            for direction in (np.inf, -np.inf):
                f = np.float32(x)
                for _ in range(3):
                    pts.add(float(f))
                    f = np.nextafter(f, np.float32(direction))
    pts |= {6.5, 7.0, 100.0, 1e30, 1e-30, 0.1, 0.3, 2.7, 5.5}
    vals = sorted(pts)
    return np.array(vals + [-v for v in vals] + [-0.0], np.float32)


def test_e2m1_encode_matches_enumeration():
    """Nearest value with exact rationals, ties to the even code, saturation
    at +-6, the sign of zero kept."""
    y = _probe_values()
    got = orc.e2m1_encode(y)
    for yy, c in zip(y.tolist(), got.tolist()):
        negative = np.signbit(np.float32(yy))
        assert c == brute.e2m1_nearest(Fraction(yy), bool(negative)), (yy, c)


def test_e2m1_ties_go_to_even_codes():
    y = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], np.float32)
    assert orc.e2m1_encode(y).tolist() == [0, 2, 2, 4, 4, 6, 6]


def test_e2m1_roundtrip_every_code():
    codes = np.arange(16, dtype=np.uint8)
    assert orc.e2m1_encode(orc.e2m1_decode(codes).astype(np.float32)).tolist() == codes.tolist()


def test_fp4_block_quant_matches_exact_rationals():
    rng = np.random.default_rng(3)
    for trial in range(6):
        x = (rng.standard_normal((16, 8)) * (10.0 ** rng.integers(-3, 4))).astype(np.float32)
        if trial == 0:
            x[3, 4] = -0.0
        codes, scales = orc.quantize_rows_fp4(x, 16)
        bc, bs = brute.quant_block_fp4_exact(np.ravel(x))
        assert float(scales[0]) == bs
        assert codes.ravel().tolist() == bc


def test_fp4_block_quant_closed_forms():
    x = np.zeros((8, 4), np.float32)
    c, s = orc.quantize_rows_fp4(x, 8)
    assert s.tolist() == [0.0] and not c.any()
    x = np.full((8, 4), -2.5, np.float32)
    c, s = orc.quantize_rows_fp4(x, 8)
    assert s[0] == np.float32(2.5 / 6) and (c == 0xF).all()        # every entry -6
    rng = np.random.default_rng(4)
    x = rng.standard_normal((64, 16)).astype(np.float32)
    c, s = orc.quantize_rows_fp4(x, 64)
    i = np.unravel_index(np.abs(x).argmax(), x.shape)
    assert orc.e2m1_decode(c[i]) == np.sign(x[i]) * 6.0
    # nearest-value property: |x/s - value| <= half the gap to the neighbouring value
    v = orc.e2m1_decode(c)
    y = x.astype(np.float64) / np.float64(s[0])
    mags = orc.e2m1_values()[:8]
    for yy, vv in zip(y.ravel(), v.ravel()):
        assert abs(abs(yy) - abs(vv)) <= np.abs(mags - abs(yy)).min() + 1e-6


def test_fp4_quantize_layout():
    d = gen.generate(2, 320, B=1, Hq=2, Hkv=1, L=96, D=16, W=8, plant=0.05)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 8, 50000)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, 8, 4, 32, fmt="fp4")
    q8 = orc.quantize(d["Q"], d["K"], d["V"], idx, 8, 8, 32, fmt="fp8")
    # queries as for FP8, keys and values in E2M1 with c_B = 6
    np.testing.assert_array_equal(qz["q_codes"], q8["q_codes"])
    np.testing.assert_array_equal(qz["q_scale"], q8["q_scale"])
    assert qz["k_codes"].max() <= 15 and qz["v_codes"].max() <= 15
    rows = qz["kq_pos"][0, 0][:32]
    kf = gen.bf16_bits_to_f32(d["K"][0, 0][rows])
    assert qz["k_scale"][0, 0, 0] == np.float32(np.abs(kf).max() / np.float32(6))
    with pytest.raises(ValueError):
        orc.quantize(d["Q"], d["K"], d["V"], idx, 8, 8, 32, fmt="fp4")


@pytest.mark.parametrize("L,D,W,ppm,block,Hq", [
    (40, 8, 6, 100000, 8, 1),
    (37, 4, 5, 200000, 5, 2),
])
def test_fp4_attention_brute_force_tiny(L, D, W, ppm, block, Hq):
    d = gen.generate(12, 321, B=1, Hq=Hq, Hkv=1, L=L, D=D, W=W, plant=0.1, outliers=(1,))
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, W, ppm)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, 4, block, fmt="fp4")
    O, Wt = orc.attention(d["Q"], d["K"], d["V"], W, 4, idx, qz, block, return_weights=True)
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
            codes, s = brute.quant_block_fp4_exact(np.ravel([Kv[p] for p in rows]))
            kc += [codes[r * D:(r + 1) * D] for r in range(len(rows))]
            ks += [s] * len(rows)
            codes, s = brute.quant_block_fp4_exact(np.ravel([Vv[p] for p in rows]))
            vc += [codes[r * D:(r + 1) * D] for r in range(len(rows))]
            vs += [s] * len(rows)
        out, wts = brute.attention_rows(Qv, Kv, Vv, L, W, 4, block, vl, qc, qs, kc, ks, vc, vs,
                                        fp4=True)
        np.testing.assert_allclose(O[h], np.array(out, np.float32), atol=1e-6, rtol=0)
        np.testing.assert_allclose(Wt[h], np.array(wts), atol=1e-12, rtol=0)


def test_fp4_hybrid_error_between_fp8_and_uniform():
    """Qualitative: one mantissa bit approximates the exact attention less
    well than FP8 codes; keeping the vertical lines and the window in full
    precision still beats FP4 everywhere (no vertical lines, W = 0)."""
    d = gen.generate(13, 322, B=1, Hq=2, Hkv=1, L=256, D=32, W=16, plant=0.02)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 16, 20000)
    exact = orc.attention(d["Q"], d["K"], d["V"], 16, 16, idx, None, 32)
    q8 = orc.quantize(d["Q"], d["K"], d["V"], idx, 16, 8, 32, fmt="fp8")
    q4 = orc.quantize(d["Q"], d["K"], d["V"], idx, 16, 4, 32, fmt="fp4")
    o8 = orc.attention(d["Q"], d["K"], d["V"], 16, 8, idx, q8, 32)
    o4 = orc.attention(d["Q"], d["K"], d["V"], 16, 4, idx, q4, 32)
    idx0, _ = orc.select_vertical(d["Q"], d["K"], 1, 0, 0)
    qu = orc.quantize(d["Q"], d["K"], d["V"], idx0, 0, 4, 32, fmt="fp4")
    ou = orc.attention(d["Q"], d["K"], d["V"], 0, 4, idx0, qu, 32)
    e8, e4, eu = (np.mean((o - exact) ** 2) for o in (o8, o4, ou))
    assert 0 < e8 < e4 < eu
