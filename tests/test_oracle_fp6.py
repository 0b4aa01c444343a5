"""Pins of the oracle's FP6 query format (OCP E2M3 query codes with
c_B = 7.5 beside E2M1 key/value codes, format "fp4q6"): the value table
against field decoding, the encoding against exact-rational enumeration,
block quantization against exact rationals and closed forms, and attention
against a scalar-loop brute force with its own quantization."""
from fractions import Fraction

import numpy as np
import pytest

import brute
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen


def test_e2m3_named_values():
    """Subnormals 0 .. 7/8 in steps of 1/8, then 1 .. 1.875 (1/8), 2 .. 3.75
    (1/4), 4 .. 7.5 (1/2); the negatives with bit 5 (code 32 is -0)."""
    v = orc.e2m3_values()
    want = [m / 8 for m in range(8)] + [1 + m / 8 for m in range(8)] + \
        [2 + m / 4 for m in range(8)] + [4 + m / 2 for m in range(8)]
    assert v[:32].tolist() == want
    assert v[32:].tolist() == [-x for x in want]
    assert np.signbit(v[32]) and not np.signbit(v[0])
    assert v.max() == 7.5 == orc.C_FP6


def test_e2m3_table_matches_field_decoding():
    for code in range(64):
        assert Fraction(float(orc.e2m3_values()[code])) == brute.e2m3_value_exact(code)


def _probe_values():
    """Every magnitude, every midpoint and their float32 neighbours (two ulps
    each way), plus saturating and tiny inputs."""
    mags = [float(brute.e2m3_value_exact(c)) for c in range(32)]
    pts = set()
    for a, b in zip(mags, mags[1:]):
        for x in (a, b, (a + b) / 2):
            for direction in (np.inf, -np.inf):
                f = np.float32(x)
                for _ in range(3):
                    pts.add(float(f))
                    f = np.nextafter(f, np.float32(direction))
    pts |= {7.6, 7.75, 8.0, 100.0, 1e30, 1e-30, 0.03, 0.0625, 0.3, 2.7, 5.1, 6.75}
    vals = sorted(pts)
    return np.array(vals + [-v for v in vals] + [-0.0], np.float32)


def test_e2m3_encode_matches_enumeration():
    """Nearest value with exact rationals, ties to the even code, saturation
    at +-7.5, the sign of zero kept."""
    y = _probe_values()
    got = orc.e2m3_encode(y)
    for yy, c in zip(y.tolist(), got.tolist()):
        negative = np.signbit(np.float32(yy))
        assert c == brute.e2m3_nearest(Fraction(yy), bool(negative)), (yy, c)


def test_e2m3_ties_go_to_even_codes():
    # midpoints: 1/16 between codes 0,1; 0.9375 between 7 (0.875) and 8 (1.0);
    # 1.9375 between 15 and 16; 3.875 between 23 and 24; 7.25 between 30 and 31
    y = np.array([0.0625, 0.1875, 0.9375, 1.9375, 3.875, 7.25], np.float32)
    assert orc.e2m3_encode(y).tolist() == [0, 2, 8, 16, 24, 30]


def test_e2m3_roundtrip_every_code():
    codes = np.arange(64, dtype=np.uint8)
    assert orc.e2m3_encode(orc.e2m3_decode(codes).astype(np.float32)).tolist() == codes.tolist()


def test_fp6_block_quant_matches_exact_rationals():
    rng = np.random.default_rng(30)
    for trial in range(6):
        x = (rng.standard_normal((16, 8)) * (10.0 ** rng.integers(-3, 4))).astype(np.float32)
        if trial == 0:
            x[3, 4] = -0.0
        codes, scales = orc.quantize_rows_fp6(x, 16)
        bc, bs = brute.quant_block_fp6_exact(np.ravel(x))
        assert float(scales[0]) == bs
        assert codes.ravel().tolist() == bc


def test_fp6_block_quant_closed_forms():
    x = np.zeros((8, 4), np.float32)
    c, s = orc.quantize_rows_fp6(x, 8)
    assert s.tolist() == [0.0] and not c.any()
    x = np.full((8, 4), -2.5, np.float32)
    c, s = orc.quantize_rows_fp6(x, 8)
    assert s[0] == np.float32(np.float32(2.5) / np.float32(7.5)) and (c == 0x3F).all()   # all -7.5
    rng = np.random.default_rng(31)
    x = rng.standard_normal((64, 16)).astype(np.float32)
    c, s = orc.quantize_rows_fp6(x, 64)
    i = np.unravel_index(np.abs(x).argmax(), x.shape)
    assert orc.e2m3_decode(c[i]) == np.sign(x[i]) * 7.5
    # nearest-value property: |x/s - value| <= the distance to every other value
    v = orc.e2m3_decode(c)
    y = x.astype(np.float64) / np.float64(s[0])
    mags = orc.e2m3_values()[:32]
    for yy, vv in zip(y.ravel(), v.ravel()):
        assert abs(abs(yy) - abs(vv)) <= np.abs(mags - abs(yy)).min() + 1e-6


def test_fp4q6_quantize_layout():
    d = gen.generate(2, 330, B=1, Hq=2, Hkv=1, L=96, D=16, W=8, plant=0.05)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 8, 50000)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, 8, 4, 32, fmt="fp4q6")
    q4 = orc.quantize(d["Q"], d["K"], d["V"], idx, 8, 4, 32, fmt="fp4")
    # keys and values exactly as for FP4; queries in E2M3 with c_B = 7.5
    for key in ("k_codes", "v_codes", "k_scale", "v_scale", "kq_pos"):
        np.testing.assert_array_equal(qz[key], q4[key])
    assert qz["q_codes"].max() <= 63
    qf = gen.bf16_bits_to_f32(d["Q"][0, 0][:32])
    assert qz["q_scale"][0, 0, 0] == np.float32(np.abs(qf).max() / np.float32(7.5))
    with pytest.raises(ValueError):
        orc.quantize(d["Q"], d["K"], d["V"], idx, 8, 8, 32, fmt="fp4q6")
    with pytest.raises(ValueError):
        orc.freeze(d["Q"], d["K"], d["V"], 1, 8, 50000, 4, 32, fmt="fp4q6")


@pytest.mark.parametrize("L,D,W,ppm,block,Hq", [
    (40, 8, 6, 100000, 8, 1),
    (37, 4, 5, 200000, 5, 2),
])
def test_fp4q6_attention_brute_force_tiny(L, D, W, ppm, block, Hq):
    d = gen.generate(14, 331, B=1, Hq=Hq, Hkv=1, L=L, D=D, W=W, plant=0.1, outliers=(1,))
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, W, ppm)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, 4, block, fmt="fp4q6")
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
            codes, s = brute.quant_block_fp6_exact(np.ravel(Qv[i:i + block]))
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
                                        fp4=True, q6=True)
        np.testing.assert_allclose(O[h], np.array(out, np.float32), atol=1e-6, rtol=0)
        np.testing.assert_allclose(Wt[h], np.array(wts), atol=1e-12, rtol=0)


def test_fp6_queries_cost_little_accuracy():
    """Qualitative: with the same E2M1 keys and values, E2M3 queries (three
    mantissa bits) approximate the exact attention less well than E4M3
    queries, within a small factor."""
    d = gen.generate(15, 332, B=1, Hq=2, Hkv=1, L=256, D=32, W=16, plant=0.02)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 16, 20000)
    exact = orc.attention(d["Q"], d["K"], d["V"], 16, 16, idx, None, 32)
    q4 = orc.quantize(d["Q"], d["K"], d["V"], idx, 16, 4, 32, fmt="fp4")
    q6 = orc.quantize(d["Q"], d["K"], d["V"], idx, 16, 4, 32, fmt="fp4q6")
    o4 = orc.attention(d["Q"], d["K"], d["V"], 16, 4, idx, q4, 32)
    o6 = orc.attention(d["Q"], d["K"], d["V"], 16, 4, idx, q6, 32)
    e4, e6 = (np.mean((o - exact) ** 2) for o in (o4, o6))
    assert 0 < e4 < e6
    # and the FP6 query error itself stays small against the exact output
    assert e6 < 4 * e4
