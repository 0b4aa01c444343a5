"""Pins of the oracle's hybrid attention (eq. prefill_hybrid with a causal
mask): exact attention where nothing is quantized, brute force on tiny
inputs, invariants, and independent dense formulations."""
import math

import numpy as np
import pytest
import torch

import brute
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen


def f64(bits):
    return torch.from_numpy(gen.bf16_bits_to_f32(bits).astype(np.float64))


def sdpa_causal(Qb, Kb, Vb):
    """Exact causal attention from torch's library routine (float64, GQA by
    repeating each KV head over its consecutive query heads)."""
    Q, K, V = f64(Qb), f64(Kb), f64(Vb)
    g = Q.shape[1] // K.shape[1]
    K = K.repeat_interleave(g, dim=1)
    V = V.repeat_interleave(g, dim=1)
    return torch.nn.functional.scaled_dot_product_attention(Q, K, V, is_causal=True).numpy()


def run(d, Hkv, W, ppm, bits, block=64, **kw):
    idx, _ = orc.select_vertical(d["Q"], d["K"], Hkv, W, ppm)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, bits, block)
    return orc.attention(d["Q"], d["K"], d["V"], W, bits, idx, qz, block, **kw), idx, qz


@pytest.mark.parametrize("W,ppm,bits", [
    (16, 50000, 16),       # bits = 16: nothing quantized
    (16, 1000000, 8),      # k = P: every prefix key is a vertical line
    (16, 1000000, 4),
    (300, 20000, 8),       # W >= L: everything is window
    (0, 0, 16),
])
def test_exact_attention_cases(W, ppm, bits):
    d = gen.generate(0, 201, B=2, Hq=4, Hkv=2, L=200, D=32, W=max(W, 1), plant=0.02)
    O, _, _ = run(d, 2, W, ppm, bits)
    ref = sdpa_causal(d["Q"], d["K"], d["V"]).reshape(O.shape)
    np.testing.assert_allclose(O, ref, atol=2e-7, rtol=0)   # float32 rounding of the fp64 result


def test_exact_attention_float64_internals():
    """Before the final float32 rounding the exact-case result equals SDPA to ~1e-12."""
    d = gen.generate(0, 202, B=1, Hq=2, Hkv=1, L=96, D=16, W=8, plant=0.02)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 8, 50000)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, 8, 16)
    ops = orc._head_operands(d["Q"], d["K"], d["V"], 0, 1, 1, 8, 16, 64, idx, qz)
    rows = np.arange(96)
    Z, Vall, pos, _, _ = orc._rows_logits(ops, rows, 16, 16, 64)
    Z = np.where(pos[None, :] <= rows[:, None], Z, -np.inf)
    E = np.exp(Z - Z.max(1, keepdims=True))
    O = (E @ Vall) / E.sum(1, keepdims=True)
    ref = sdpa_causal(d["Q"], d["K"], d["V"])[0, 1]
    np.testing.assert_allclose(O, ref, atol=1e-12, rtol=0)


@pytest.mark.parametrize("L,D,W,ppm,bits,block,Hq", [
    (12, 4, 3, 200000, 8, 4, 2),
    (16, 8, 4, 150000, 4, 2, 2),
    (10, 4, 0, 0, 8, 3, 1),            # uniform quantization, no window
    (14, 8, 5, 0, 8, 4, 1),            # window only
    (9, 4, 2, 1000000, 8, 2, 1),       # every prefix key vertical
])
def test_brute_force_tiny(L, D, W, ppm, bits, block, Hq):
    d = gen.generate(9, 203, B=1, Hq=Hq, Hkv=1, L=L, D=D, W=max(W, 1), plant=0.1, outliers=(1,))
    O, idx, qz = run(d, 1, W, ppm, bits, block, return_weights=True)
    O, Wt = O
    c = orc.code_bound(bits)
    P = max(0, L - W)
    vl = idx[0, 0].tolist()
    qpos = [p for p in range(P) if p not in set(vl)]
    for h in range(Hq):
        Qv = gen.bf16_bits_to_f32(d["Q"][0, h]).astype(np.float64).tolist()
        Kv = gen.bf16_bits_to_f32(d["K"][0, 0]).astype(np.float64).tolist()
        Vv = gen.bf16_bits_to_f32(d["V"][0, 0]).astype(np.float64).tolist()
        # brute quantization (exact rationals), independent of the oracle
        qc, qs = [], []
        for i in range(0, L, block):
            codes, s = brute.quant_block_exact(np.ravel(Qv[i:i + block]), 127)
            qc += [codes[r * D:(r + 1) * D] for r in range(min(block, L - i))]
            qs.append(s)
        kc, ks, vc, vs = [], [], [], []
        for i in range(0, len(qpos), block):
            rows = qpos[i:i + block]
            codes, s = brute.quant_block_exact(np.ravel([Kv[p] for p in rows]), c)
            kc += [codes[r * D:(r + 1) * D] for r in range(len(rows))]
            ks += [s] * len(rows)
            codes, s = brute.quant_block_exact(np.ravel([Vv[p] for p in rows]), c)
            vc += [codes[r * D:(r + 1) * D] for r in range(len(rows))]
            vs += [s] * len(rows)
        out, wts = brute.attention_rows(Qv, Kv, Vv, L, W, bits, block, vl,
                                        qc, qs, kc, ks, vc, vs)
        np.testing.assert_allclose(O[h], np.array(out, np.float32), atol=1e-6, rtol=0)
        np.testing.assert_allclose(Wt[h], np.array(wts), atol=1e-12, rtol=0)


def test_invariants_rows_sum_to_one_and_causal():
    d = gen.generate(2, 204, B=1, Hq=2, Hkv=1, L=150, D=16, W=10, plant=0.05)
    (O, Wt), idx, qz = run(d, 1, 10, 50000, 8, 16, return_weights=True)
    np.testing.assert_allclose(Wt.sum(axis=2), 1.0, atol=1e-13)
    upper = np.triu(np.ones((150, 150), bool), k=1)
    assert np.all(Wt[:, upper] == 0.0)
    assert np.all(Wt[:, ~upper] > 0.0)


def test_first_row_is_value_of_key_zero():
    d = gen.generate(3, 205, B=1, Hq=1, Hkv=1, L=130, D=8, W=10, plant=0.0)
    for ppm in (0, 1000000):
        O, idx, qz = run(d, 1, 10, ppm, 8, 16)
        if 0 in idx[0, 0]:
            v0 = gen.bf16_bits_to_f32(d["V"][0, 0, 0])
        else:
            v0 = qz["v_scale"][0, 0, 0].astype(np.float64) * qz["v_codes"][0, 0, 0]
        np.testing.assert_array_equal(O[0, 0], np.float32(v0))


def test_stage_level_causality():
    """With selection and quantization outputs held fixed, changing inputs at
    rows after t leaves row t bit-identical."""
    d = gen.generate(4, 206, B=1, Hq=2, Hkv=1, L=160, D=16, W=12, plant=0.05)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 12, 50000)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, 12, 8, 16)
    O1 = orc.attention(d["Q"], d["K"], d["V"], 12, 8, idx, qz, 16)
    t = 95
    Q2, K2, V2 = d["Q"].copy(), d["K"].copy(), d["V"].copy()
    rng = np.random.default_rng(0)
    for A in (Q2, K2, V2):
        A[:, :, t + 1:] = gen.f32_to_bf16_bits(rng.standard_normal(A[:, :, t + 1:].shape).astype(np.float32))
    qz2 = dict(qz)
    for key, A in (("q_codes", qz["q_codes"]),):
        B2 = A.copy()
        B2[:, :, t + 1:] = rng.integers(-127, 128, size=B2[:, :, t + 1:].shape)
        qz2[key] = B2
    O2 = orc.attention(Q2, K2, V2, 12, 8, idx, qz2, 16)
    np.testing.assert_array_equal(O1[:, :t + 1], O2[:, :t + 1])
    assert np.any(O1[:, t + 1:] != O2[:, t + 1:])


def _dequant_dense(Qb, Kb, Vb, W, bits, block, idx, fake_q):
    """Independent dense formulation: fake-quantize (quantize then dequantize)
    Q and the compacted K/V with explicit block loops, then one masked softmax
    over original key positions with torch."""
    B, Hq, L, D = Qb.shape
    P = max(0, L - W)
    c = 127 if bits == 8 else 7
    Q, K, V = f64(Qb)[0], f64(Kb)[0], f64(Vb)[0]
    out = []
    for h in range(Hq):
        Kh, Vh = K[0].clone(), V[0].clone()
        vl = set(idx[0, 0].tolist())
        qpos = [p for p in range(P) if p not in vl]
        Kq, Vq = Kh.clone(), Vh.clone()
        for i in range(0, len(qpos), block):
            rows = qpos[i:i + block]
            for src, dst in ((Kh, Kq), (Vh, Vq)):
                blk = src[rows].float()
                s = (blk.abs().max() / c).float()
                codes = torch.zeros_like(blk) if s == 0 else torch.clamp(torch.round(blk / s), -c, c)
                dst[rows] = codes.double() * s.double()
        Qh = Q[h].clone()
        Qhat = Qh.clone()
        for i in range(0, L, block):
            blk = Qh[i:i + block].float()
            s = (blk.abs().max() / 127).float()
            codes = torch.zeros_like(blk) if s == 0 else torch.clamp(torch.round(blk / s), -127, 127)
            Qhat[i:i + block] = codes.double() * s.double()
        alpha = 1.0 / math.sqrt(D)
        Zq = alpha * (Qhat @ Kq.T)
        Zf = alpha * (Qh @ Kh.T)
        isq = torch.zeros(L, dtype=torch.bool)
        isq[qpos] = True
        Z = torch.where(isq[None, :], Zq, Zf)
        Vall = torch.where(isq[:, None], Vq, Vh)
        mask = torch.ones(L, L, dtype=torch.bool).tril()
        Z = Z.masked_fill(~mask, -math.inf)
        out.append((torch.softmax(Z, dim=1) @ Vall).numpy())
    return np.stack(out)


@pytest.mark.parametrize("W,ppm,bits", [(24, 0, 8), (24, 0, 4), (0, 0, 8), (24, 40000, 8), (7, 90000, 4)])
def test_matches_dense_fake_quant_formulation(W, ppm, bits):
    """Window-only (budget 0), uniform (W = 0) and hybrid cases against a
    dense fake-quantization formulation (dequantized values, library softmax)."""
    L, D, block = 200, 32, 32
    d = gen.generate(5, 207, B=1, Hq=3, Hkv=1, L=L, D=D, W=max(W, 1), plant=0.03)
    O, idx, qz = run(d, 1, W, ppm, bits, block)
    ref = _dequant_dense(d["Q"], d["K"], d["V"], W, bits, block, idx, True)
    np.testing.assert_allclose(O[:, :], ref.astype(np.float32), atol=1e-6, rtol=0)


def test_rows_and_heads_subset_consistent():
    d = gen.generate(6, 208, B=2, Hq=4, Hkv=2, L=300, D=16, W=20, plant=0.02)
    Ofull, idx, qz = run(d, 2, 20, 30000, 8, 64)
    rows = np.array([0, 5, 279, 280, 299])
    heads = [(1, 3), (0, 1)]
    Osub = orc.attention(d["Q"], d["K"], d["V"], 20, 8, idx, qz, 64, heads=heads, rows=rows)
    np.testing.assert_array_equal(Osub[0], Ofull[1 * 4 + 3][rows])
    np.testing.assert_array_equal(Osub[1], Ofull[0 * 4 + 1][rows])


def test_mse_ordering_qualitative():
    """Retaining vertical lines and a window lowers the error against exact
    attention, and more retention lowers it further (cf. the window and ratio
    ablations and the MSE comparison of Section 2.2)."""
    d = gen.generate(0, 209, B=1, Hq=4, Hkv=1, L=1024, D=128, W=64, plant=0.01)
    exact = sdpa_causal(d["Q"], d["K"], d["V"])[0]

    def mse(W, ppm, bits):
        O, _, _ = run(d, 1, W, ppm, bits)
        return float(np.mean((O - exact) ** 2))
    uniform4 = mse(0, 0, 4)
    hybrid4 = mse(64, 20000, 4)
    assert hybrid4 < uniform4
    assert mse(64, 50000, 4) < mse(64, 5000, 4)
    assert mse(128, 20000, 4) < mse(16, 20000, 4)
    assert mse(64, 20000, 8) < hybrid4
