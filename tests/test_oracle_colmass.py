"""Pins of the oracle's exact column-mass selector (eq. vl_score, eq. vl_topk):
the attention mass of the tail queries on every key."""
import math

import numpy as np
import pytest

import brute
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen


def test_mass_sums_to_the_number_of_query_rows():
    """Each considered softmax row sums to 1: S over all keys sums to g * t."""
    L, D, W, Hq, Hkv = 150, 16, 24, 4, 2
    d = gen.generate(1, 800, B=2, Hq=Hq, Hkv=Hkv, L=L, D=D, W=W, plant=0.05)
    S = orc.column_mass(d["Q"], d["K"], Hkv, W)
    np.testing.assert_allclose(S.sum(-1), (Hq // Hkv) * min(W, L), rtol=1e-12)
    assert np.all(S >= 0)


@pytest.mark.parametrize("L,D,W,ppm,Hq,Hkv", [(14, 4, 4, 250000, 2, 1), (11, 8, 3, 300000, 4, 2)])
def test_colmass_brute_force_tiny(L, D, W, ppm, Hq, Hkv):
    """Scalar loops with math.exp / math.fsum, ranking by (score desc, position asc)."""
    d = gen.generate(2, 801, B=1, Hq=Hq, Hkv=Hkv, L=L, D=D, W=W, plant=0.1)
    idx, S = orc.select_vertical_colmass(d["Q"], d["K"], Hkv, W, ppm)
    g = Hq // Hkv
    t = min(W, L)
    P = L - W
    k = orc.sizes(L, W, ppm)["k"]
    for j in range(Hkv):
        Kv = [[brute.bf16_value(x) for x in row] for row in d["K"][0, j]]
        col = [0.0] * L
        for r in range(g):
            for i in range(L - t, L):
                qv = [brute.bf16_value(x) for x in d["Q"][0, j * g + r, i]]
                z = [math.fsum(qv[e] * Kv[p][e] for e in range(D)) / math.sqrt(D)
                     for p in range(i + 1)]
                m = max(z)
                w = [math.exp(x - m) for x in z]
                den = math.fsum(w)
                for p in range(i + 1):
                    col[p] += w[p] / den
        np.testing.assert_allclose(S[0, j], col[:P], rtol=1e-12, atol=1e-15)
        order = sorted(range(P), key=lambda p: (-col[p], p))[:k]
        assert idx[0, j].tolist() == sorted(order)


def test_colmass_invariant_to_a_common_key_shift():
    """Adding one vector c to every key adds q . c to each softmax row: the
    column mass does not change.  Integer-valued inputs keep the shift exact
    in bf16."""
    L, D, W = 120, 8, 16
    rng = np.random.default_rng(5)
    Q = np.round(rng.standard_normal((1, 2, L, D)) * 2).astype(np.float32)
    K = np.round(rng.standard_normal((1, 1, L, D)) * 2).astype(np.float32)
    c = np.round(rng.standard_normal(D) * 3).astype(np.float32)
    S1 = orc.column_mass(gen.f32_to_bf16_bits(Q), gen.f32_to_bf16_bits(K), 1, W)
    S2 = orc.column_mass(gen.f32_to_bf16_bits(Q), gen.f32_to_bf16_bits(K + c), 1, W)
    np.testing.assert_allclose(S1, S2, rtol=1e-9, atol=1e-12)
    S3 = orc.column_mass(gen.f32_to_bf16_bits(Q), gen.f32_to_bf16_bits(K * 2), 1, W)
    assert np.abs(S1 - S3).max() > 1e-3          # scaling the keys is not an invariance


def test_colmass_picks_a_dominant_key_and_respects_the_budget():
    L, D, W, ppm = 200, 16, 32, 10000
    d = gen.generate(4, 803, B=1, Hq=2, Hkv=1, L=L, D=D, W=W, plant=0.0)
    K = gen.bf16_bits_to_f32(d["K"])
    Q = gen.bf16_bits_to_f32(d["Q"])
    u = Q[0, :, L - W:].sum(axis=(0, 1))
    K[0, 0, 77] = 40.0 * u / np.linalg.norm(u)             # every tail query looks at key 77
    d["K"] = gen.f32_to_bf16_bits(K)
    idx, S = orc.select_vertical_colmass(d["Q"], d["K"], 1, W, ppm)
    assert idx.shape[-1] == orc.sizes(L, W, ppm)["k"] == 2
    assert 77 in idx[0, 0].tolist()
    assert S[0, 0, 77] == S[0, 0].max()
