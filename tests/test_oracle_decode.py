"""Pins of the oracle's decode path: Algorithm 4 (Freeze), the staging buffer
and its merge, and Algorithm 3 (decode attention over the four buffers)."""
import math

import numpy as np
import pytest

import brute
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen


def _prefill(seed, B, Hq, Hkv, N, D, W):
    return gen.generate(seed, 600 + seed, B=B, Hq=Hq, Hkv=Hkv, L=N, D=D, W=max(W, 1), plant=0.05)


def _new_rows(rng, B, H, D):
    return gen.f32_to_bf16_bits(rng.standard_normal((B, H, D)).astype(np.float32))


def _all_positions(cache, bj):
    return orc.decode_keys(cache, bj)[2]


@pytest.mark.parametrize("fmt,bits", [("int", 8), ("int", 4), ("fp8", 8), ("fp4", 4)])
def test_freeze_partition_and_reuse_of_prefill_steps(fmt, bits):
    N, W, ppm = 400, 96, 50000
    d = _prefill(1, 2, 4, 2, N, 16, W)
    c = orc.freeze(d["Q"], d["K"], d["V"], 2, W, ppm, bits, fmt=fmt)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 2, W, ppm)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, bits, 64, fmt)
    for b in range(2):
        for j in range(2):
            bj = b * 2 + j
            pos = _all_positions(c, bj)
            assert sorted(pos.tolist()) == list(range(N))           # each token exactly once
            np.testing.assert_array_equal(np.concatenate(c["k_blocks"][bj]), qz["k_codes"][b, j])
            np.testing.assert_array_equal(np.concatenate(c["v_blocks"][bj]), qz["v_codes"][b, j])
            np.testing.assert_array_equal(c["vl_k"][bj], d["K"][b, j][idx[b, j]])
            np.testing.assert_array_equal(np.stack(c["win_v"][bj]), d["V"][b, j][N - W:])
            assert c["st_k"][bj] == []


def test_decode_without_quantized_keys_is_exact_attention():
    """budget 100%: every prefix key is a vertical line, nothing is quantized;
    decode attention must equal plain softmax attention over all tokens,
    computed here independently (scalar loop, math.exp)."""
    N, W, D = 130, 64, 8
    d = _prefill(2, 1, 2, 1, N, D, W)
    c = orc.freeze(d["Q"], d["K"], d["V"], 1, W, 1000000, 8)
    rng = np.random.default_rng(3)
    Kall = [d["K"][0, 0, p] for p in range(N)]
    Vall = [d["V"][0, 0, p] for p in range(N)]
    for step in range(70):                      # crosses one merge (Ws = 64)
        kn, vn = _new_rows(rng, 1, 1, D), _new_rows(rng, 1, 1, D)
        orc.decode_append(c, kn, vn)
        Kall.append(kn[0, 0])
        Vall.append(vn[0, 0])
        if step in (0, 63, 64, 69):
            # exact only while no merged block exists (merges quantize old window rows)
            q = _new_rows(rng, 1, 2, D)
            O = orc.decode_attention(q, c)
            if len(c["k_blocks"][0]) == 0:
                for h in range(2):
                    qv = [brute.bf16_value(x) for x in q[0, h]]
                    zs = [math.fsum(qv[e] * brute.bf16_value(k[e]) for e in range(D)) / math.sqrt(D)
                          for k in Kall]
                    m = max(zs)
                    ws = [math.exp(z - m) for z in zs]
                    ref = [math.fsum(w * brute.bf16_value(v[e]) for w, v in zip(ws, Vall)) /
                           math.fsum(ws) for e in range(D)]
                    np.testing.assert_allclose(O[0, h], np.float32(ref), atol=2e-6, rtol=0)
    assert len(c["k_blocks"][0]) == 1                # the merge happened at the 65th token


@pytest.mark.parametrize("fmt,bits", [("int", 8), ("int", 4), ("fp8", 8), ("fp4", 4)])
def test_merge_quantizes_the_oldest_window_block(fmt, bits):
    N, W, D = 300, 80, 8
    d = _prefill(4, 1, 2, 1, N, D, W)
    c = orc.freeze(d["Q"], d["K"], d["V"], 1, W, 30000, bits, fmt=fmt)
    nb0 = len(c["k_blocks"][0])
    oldest_k = np.stack(c["win_k"][0][:64])
    oldest_pos = c["win_pos"][0][:64]
    rng = np.random.default_rng(5)
    added = []
    for _ in range(65):
        kn, vn = _new_rows(rng, 1, 1, D), _new_rows(rng, 1, 1, D)
        orc.decode_append(c, kn, vn)
        added.append(kn[0, 0])
    assert len(c["k_blocks"][0]) == nb0 + 1
    assert len(c["win_k"][0]) == W and len(c["st_k"][0]) == 1
    assert list(c["q_pos"][0][-1]) == oldest_pos
    assert sorted(_all_positions(c, 0).tolist()) == list(range(N + 65))
    # the new block: exact-rational quantization of the 64 evicted rows
    x = gen.bf16_bits_to_f32(oldest_k).ravel()
    if fmt == "fp8":
        codes, s = brute.quant_block_fp8_exact(x)
    elif fmt == "fp4":
        codes, s = brute.quant_block_fp4_exact(x)
    else:
        codes, s = brute.quant_block_exact(x, orc.code_bound(bits))
    assert np.ravel(c["k_blocks"][0][-1]).tolist() == codes
    assert float(c["k_scales"][0][-1]) == s
    # the 64 staged tokens joined the window, newest last
    np.testing.assert_array_equal(np.stack(c["win_k"][0][-64:]), np.stack(added[:64]))


@pytest.mark.parametrize("fmt,bits", [("int", 8), ("fp8", 8), ("fp4", 4)])
def test_decode_attention_brute_force_tiny(fmt, bits):
    """Scalar-loop attention over the four buffers, dequantizing every code
    from its fields / integer value, with exact sums."""
    N, W, D, g = 150, 64, 4, 2
    d = _prefill(6, 1, g, 1, N, D, W)
    c = orc.freeze(d["Q"], d["K"], d["V"], 1, W, 40000, bits, fmt=fmt)
    rng = np.random.default_rng(7)
    for _ in range(66):
        orc.decode_append(c, _new_rows(rng, 1, 1, D), _new_rows(rng, 1, 1, D))
    q = _new_rows(rng, 1, g, D)
    O = orc.decode_attention(q, c)

    def cval(code):
        if fmt == "fp4":
            return float(brute.e2m1_value_exact(code))
        return float(brute.e4m3_value_exact(code)) if fmt == "fp8" else int(code)
    keys, vals = [], []
    for kc, vc, ks, vs, pos in zip(c["k_blocks"][0], c["v_blocks"][0], c["k_scales"][0],
                                   c["v_scales"][0], c["q_pos"][0]):
        for n in range(len(pos)):
            keys.append([float(ks) * cval(x) for x in kc[n]])
            vals.append([float(vs) * cval(x) for x in vc[n]])
    for kk, vv in ((c["vl_k"][0], c["vl_v"][0]), (c["win_k"][0], c["win_v"][0]),
                   (c["st_k"][0], c["st_v"][0])):
        for kr, vr in zip(kk, vv):
            keys.append([brute.bf16_value(x) for x in kr])
            vals.append([brute.bf16_value(x) for x in vr])
    assert len(keys) == N + 66
    for h in range(g):
        qv = [brute.bf16_value(x) for x in q[0, h]]
        zs = [math.fsum(qv[e] * k[e] for e in range(D)) / math.sqrt(D) for k in keys]
        m = max(zs)
        ws = [math.exp(z - m) for z in zs]
        ref = [math.fsum(w * v[e] for w, v in zip(ws, vals)) / math.fsum(ws) for e in range(D)]
        np.testing.assert_allclose(O[0, h], np.float32(ref), atol=2e-6, rtol=0)


def test_decode_weights_sum_to_one_and_key_order_irrelevant():
    N, W, D = 200, 64, 8
    d = _prefill(8, 1, 4, 1, N, D, W)
    c = orc.freeze(d["Q"], d["K"], d["V"], 1, W, 20000, 8)
    q = _new_rows(np.random.default_rng(9), 1, 4, D)
    O1 = orc.decode_attention(q, c)
    # reversing the window order and the block order changes nothing
    c["win_k"][0] = c["win_k"][0][::-1]
    c["win_v"][0] = c["win_v"][0][::-1]
    for name in ("k_blocks", "v_blocks", "k_scales", "v_scales", "q_pos"):
        c[name][0] = c[name][0][::-1]
    O2 = orc.decode_attention(q, c)
    np.testing.assert_allclose(O1, O2, atol=1e-6, rtol=0)
    # a value shift by a constant row shifts every output by that row
    c2 = orc.freeze(d["Q"], d["K"], d["V"] * 0, 1, W, 20000, 8)   # all-zero values
    assert np.all(orc.decode_attention(q, c2) == 0)


def test_freeze_domain():
    d = _prefill(10, 1, 2, 1, 100, 8, 64)
    with pytest.raises(ValueError):
        orc.freeze(d["Q"], d["K"], d["V"], 1, 32, 10000, 8)        # W < Ws
    with pytest.raises(ValueError):
        orc.freeze(d["Q"], d["K"], d["V"], 1, 128, 10000, 8)       # N < W
    with pytest.raises(ValueError):
        orc.freeze(d["Q"], d["K"], d["V"], 1, 64, 10000, 16)       # nothing quantized


@pytest.mark.parametrize("fmt,bits", [("int", 8), ("fp4", 4)])
def test_merge_with_a_two_block_staging_buffer(fmt, bits):
    """Staging capacity 128 (the memory-overhead example of the paper): the
    129th token merges the 128 oldest window tokens into two blocks, each
    quantized on its own (exact rationals), oldest first."""
    N, W, D = 300, 128, 8
    d = _prefill(11, 1, 2, 1, N, D, W)
    c = orc.freeze(d["Q"], d["K"], d["V"], 1, W, 30000, bits, fmt=fmt, staging=128)
    nb0 = len(c["k_blocks"][0])
    oldest_k = np.stack(c["win_k"][0][:128])
    oldest_pos = c["win_pos"][0][:128]
    rng = np.random.default_rng(12)
    added = []
    for step in range(129):
        kn, vn = _new_rows(rng, 1, 1, D), _new_rows(rng, 1, 1, D)
        orc.decode_append(c, kn, vn)
        added.append(kn[0, 0])
        if step < 128:
            assert len(c["k_blocks"][0]) == nb0           # no merge before the 129th token
    assert len(c["k_blocks"][0]) == nb0 + 2
    assert len(c["win_k"][0]) == W and len(c["st_k"][0]) == 1
    assert sorted(_all_positions(c, 0).tolist()) == list(range(N + 129))
    for i in range(2):
        x = gen.bf16_bits_to_f32(oldest_k[64 * i:64 * (i + 1)]).ravel()
        codes, s = brute.quant_block_fp4_exact(x) if fmt == "fp4" else \
            brute.quant_block_exact(x, orc.code_bound(bits))
        assert np.ravel(c["k_blocks"][0][nb0 + i]).tolist() == codes
        assert float(c["k_scales"][0][nb0 + i]) == s
        assert list(c["q_pos"][0][nb0 + i]) == oldest_pos[64 * i:64 * (i + 1)]
    np.testing.assert_array_equal(np.stack(c["win_k"][0]), np.stack(added[:128]))


def test_staging_capacity_domain():
    d = _prefill(13, 1, 2, 1, 300, 8, 128)
    for bad in (0, 32, 100, 192):                           # not a block multiple, or > W
        with pytest.raises(ValueError):
            orc.freeze(d["Q"], d["K"], d["V"], 1, 128, 10000, 8, staging=bad)
