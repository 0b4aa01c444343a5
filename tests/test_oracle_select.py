"""Pins of the oracle's selection (Algorithm 1) against closed forms, brute
force and exact integer arithmetic."""
import numpy as np
import pytest

import brute
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


@pytest.mark.parametrize("L,W,ppm,P,k,nQ,nkv", [
    # Closed forms of Algorithm 1: P = L - W, k = min(P, max(1, ceil(P*r))).
    (1024, 64, 20000, 960, 20, 940, 15),          # ceil(19.2) = 20; 940 = 14*64 + 44
    (8192, 128, 20000, 8064, 162, 7902, 124),     # ceil(161.28) = 162
    (32768, 256, 10000, 32512, 326, 32186, 503),  # ceil(325.12) = 326; 32186 = 502*64 + 58
    (131072, 512, 5000, 130560, 653, 129907, 2030),  # ceil(652.8) = 653
    (16384, 256, 5000, 16128, 81, 16047, 251),    # ceil(80.64) = 81
    (16384, 256, 20000, 16128, 323, 15805, 247),  # ceil(322.56) = 323
    (16384, 256, 50000, 16128, 807, 15321, 240),  # ceil(806.4) = 807
    (100, 10, 1, 90, 1, 89, 2),                   # tiny ratio still keeps one line
    (100, 10, 1000000, 90, 90, 0, 0),             # r = 1 keeps the whole prefix
    (100, 100, 50000, 0, 0, 0, 0),                # window covers everything: P = 0
    (100, 200, 50000, 0, 0, 0, 0),
    (100, 10, 0, 90, 0, 90, 2),                   # budget 0: window-only retention
    (1000, 0, 20000, 1000, 20, 980, 16),
])
def test_sizes_closed_form(L, W, ppm, P, k, nQ, nkv):
    s = orc.sizes(L, W, ppm)
    assert (s["P"], s["k"], s["nQ"], s["n_kvblk"]) == (P, k, nQ, nkv)
    assert s["n_qblk"] == -(-L // 64)


def test_topk_matches_rank_count():
    rng = np.random.default_rng(1)
    for trial in range(40):
        n = int(rng.integers(1, 40))
        S = rng.integers(-3, 4, size=n).astype(np.float32)        # many ties
        if trial % 3 == 0:
            S[rng.random(n) < 0.3] = np.float32(-0.0)             # signed zeros
        k = int(rng.integers(1, n + 1))
        got = orc.topk_ascending(S[None], k)[0].tolist()
        assert got == brute.topk_by_rank(S, k)


def test_topk_signed_zero_tie_lowest_index():
    S = np.array([-0.0, 0.0, -0.0, -1.0, 0.0], dtype=np.float32)
    assert orc.topk_ascending(S[None], 2)[0].tolist() == [0, 1]
    assert orc.topk_ascending(S[None], 4)[0].tolist() == [0, 1, 2, 4]


@pytest.mark.parametrize("B,Hq,Hkv,L,D,W,ppm", [
    (1, 1, 1, 50, 8, 8, 100000),
    (2, 4, 2, 70, 16, 16, 60000),
    (1, 6, 2, 33, 8, 40, 200000),     # W > L: t = L, P = 0
    (1, 5, 1, 64, 4, 3, 500000),      # g = 5
    (1, 4, 1, 129, 128, 17, 30000),   # D = 128: the full pinned tree
])
def test_select_integer_inputs_exact(B, Hq, Hkv, L, D, W, ppm):
    """Small-integer bf16 inputs make every float32 operation exact, so the
    result must equal int64 arithmetic ranked by (score desc, position asc)."""
    rng = np.random.default_rng([B, Hq, L, D])
    Qi = rng.integers(-3, 4, size=(B, Hq, L, D))
    Ki = rng.integers(-2, 3, size=(B, Hkv, L, D))
    Qb = gen.f32_to_bf16_bits(Qi.astype(np.float32))
    Kb = gen.f32_to_bf16_bits(Ki.astype(np.float32))
    idx, S = orc.select_vertical(Qb, Kb, Hkv, W, ppm)
    k = orc.sizes(L, W, ppm)["k"]
    assert idx.shape == (B, Hkv, k)
    if k:
        np.testing.assert_array_equal(idx, brute.int_select(Qi, Ki, Hkv, W, k))


def test_select_integer_scores_equal_int64():
    rng = np.random.default_rng(7)
    B, Hq, Hkv, L, D, W = 1, 4, 2, 90, 128, 20
    Qi = rng.integers(-2, 3, size=(B, Hq, L, D))
    Ki = rng.integers(-2, 3, size=(B, Hkv, L, D))
    Qf = Qi.astype(np.float32)
    qsum = orc.tail_proxy(Qf, Hkv, W)
    S = orc.scores(qsum, Ki.astype(np.float32), L - W)
    for j in range(Hkv):
        qs = Qi[0, 2 * j:2 * j + 2, L - W:, :].sum(axis=(0, 1))
        np.testing.assert_array_equal(S[0, j], (Ki[0, j, :L - W] @ qs).astype(np.float32))


def test_select_invariants_generated():
    d = gen.generate(3, 101, B=2, Hq=8, Hkv=2, L=700, D=128, W=48, plant=0.02)
    idx, S = orc.select_vertical(d["Q"], d["K"], 2, 48, 30000)
    P, k = 652, 20
    assert idx.shape == (2, 2, k)
    for b in range(2):
        for j in range(2):
            v = idx[b, j]
            assert np.all(np.diff(v) > 0) and v[0] >= 0 and v[-1] < P
            # every chosen score >= every unchosen score
            rest = np.setdiff1d(np.arange(P), v)
            assert S[b, j, v].min() >= S[b, j, rest].max()


def test_planted_lines_recovered():
    """Sanity: most planted vertical lines (aligned with the tail proxy) are
    found; the x10 outlier channels add score noise, so recall is not 1."""
    d = gen.generate_workload(gen.SMALL, seed=0)
    idx, _ = orc.select_vertical(d["Q"], d["K"], 1, 64, 20000)
    planted = set(d["planted"][0].tolist())
    P = 960
    planted_prefix = {p for p in planted if p < P}
    hit = len(planted_prefix & set(idx[0, 0].tolist()))
    assert hit >= 0.8 * len(planted_prefix)


def test_pinned_tree_order_matters():
    """The fold order is a contract: a sequential sum gives different bits on
    generic data, so a kernel that reorders would be caught."""
    rng = np.random.default_rng(5)
    prod = rng.standard_normal((2000, 128)).astype(np.float32)
    seq = np.zeros(2000, np.float32)
    for d in range(128):
        seq = seq + prod[:, d]
    assert np.any(orc.fold_sum(prod) != seq)
    # and the fold equals an explicit pairing written out for D = 4
    v = np.array([[1e8, 1.0, -1e8, 1.0]], dtype=np.float32)
    # (v0 + v2) + (v1 + v3) = 0 + 2 = 2
    assert orc.fold_sum(v)[0] == np.float32(2.0)


@pytest.mark.parametrize("kind", gen.TIE_KINDS)
def test_tie_inputs_tie_at_threshold(kind):
    """The tie inputs (used by the GPU tie test) really put many exact ties,
    and signed zeros, at the k-th largest score, spread over the prefix; on
    them the oracle's selection equals int64 scores ranked by rank counting
    with -0 == +0 (lowest position wins)."""
    B, Hq, Hkv, L, W, ppm = 1, 8, 4, 2048, 64, 20000
    k = orc.sizes(L, W, ppm)["k"]
    P = L - W
    d = gen.tie_inputs(11, B, Hq, Hkv, L, W, k, kind)
    idx, S = orc.select_vertical(d["Q"], d["K"], Hkv, W, ppm)
    Qi = gen.bf16_bits_to_f32(d["Q"]).astype(np.int64)
    Ki = gen.bf16_bits_to_f32(d["K"]).astype(np.int64)
    g = Hq // Hkv
    for j in range(Hkv):
        c = Qi[0, j * g:(j + 1) * g, L - W:, :].sum(axis=(0, 1))
        Sint = Ki[0, j, :P] @ c
        np.testing.assert_array_equal(S[0, j], Sint.astype(np.float32))
        T = np.sort(Sint)[::-1][k - 1]
        n_gt, n_eq = int((Sint > T).sum()), int((Sint == T).sum())
        assert n_eq > k - n_gt >= 1                   # ties at the threshold must be split
        eq_pos = np.nonzero(Sint == T)[0]
        assert eq_pos.min() < P // 8 and eq_pos.max() > P - P // 8
        if kind != "positive":
            assert T == 0
            bits = S[0, j].view(np.uint32)
            zero_pos = np.nonzero(Sint == 0)[0]
            assert np.any(bits[zero_pos] == 0x80000000) and np.any(bits[zero_pos] == 0)
        # rank counting: p is chosen iff fewer than k keys beat it
        beat = np.array([(Sint > Sint[p]).sum() + (Sint[:p] == Sint[p]).sum() for p in range(P)])
        np.testing.assert_array_equal(idx[0, j], np.nonzero(beat < k)[0])
