"""Seeded synthetic inputs for the HyQuant prefill path.

This module only draws inputs; it holds none of the method's arithmetic
(no selection, quantization or attention).  Both the HIP path and the CPU
oracle consume exactly the bf16 bit patterns produced here.

Workload recipe (stands in for real-model activations, which are not
available): Q, K, V ~ N(0, 1) drawn as float32 and rounded to bf16; a set
of "vertical-line" key rows per KV head (position 0 plus a fraction of
random positions) gets 4 * (unit direction of the summed tail queries of
that KV head's query group) added; finally four fixed K channels are scaled
by 10 on every key (outlier channels, the case per-block quantization
handles worst).  Shapes follow the paper's models (GQA 32q/8kv and 40q/8kv,
head_dim 128, Section 5.1 and the configuration table of App. B).
"""
from __future__ import annotations

import numpy as np

OUTLIER_CHANNELS = (3, 47, 85, 122)

# The five workloads, named by shape: batch, heads, length, window, vertical
# budget (parts per million of the non-window prefix), K/V bit-width, the
# planted vertical-line fraction, and the generator stream that separates
# workloads drawn with the same seed.
WORKLOADS = {
    "gqa1q1kv_B1_L1024": dict(stream=1, B=1, Hq=1, Hkv=1, L=1024, D=128, W=64,
                              budget_ppm=20000, bits=8, plant=0.01),
    "gqa32q8kv_B1_L8192": dict(stream=2, B=1, Hq=32, Hkv=8, L=8192, D=128, W=128,
                               budget_ppm=20000, bits=8, plant=0.01),
    "gqa32q8kv_B1_L32768": dict(stream=3, B=1, Hq=32, Hkv=8, L=32768, D=128, W=256,
                                budget_ppm=10000, bits=8, plant=0.01),
    "gqa32q8kv_B1_L131072": dict(stream=4, B=1, Hq=32, Hkv=8, L=131072, D=128, W=512,
                                 budget_ppm=5000, bits=8, plant=0.01),
    "gqa40q8kv_B4_L16384": dict(stream=5, B=4, Hq=40, Hkv=8, L=16384, D=128, W=256,
                                budget_ppm=20000, bits=8, plant=0.05),
}
SMALL = "gqa1q1kv_B1_L1024"
GQA_8K = "gqa32q8kv_B1_L8192"
GQA_32K = "gqa32q8kv_B1_L32768"      # the benchmarked prefill workload
GQA_128K = "gqa32q8kv_B1_L131072"
BATCH4_16K = "gqa40q8kv_B4_L16384"
# The batch-4 16k workload is run as a sweep over these two axes.
BATCH4_BUDGETS = (5000, 20000, 50000)
BATCH4_BITS = (8, 4)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round-to-nearest-even); returns uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.ascontiguousarray(b).astype(np.uint32) << np.uint32(16)).view(np.float32)


def generate(seed: int, stream: int, B: int, Hq: int, Hkv: int, L: int, D: int,
             W: int, plant: float, outliers=OUTLIER_CHANNELS, **_unused):
    """Draw one seeded input set.

    Returns a dict with uint16 (bf16 bit pattern) arrays ``Q`` [B,Hq,L,D],
    ``K`` and ``V`` [B,Hkv,L,D], and ``planted``: a list over (b, j) of the
    sorted planted key positions.  ``stream`` separates workloads that share a
    seed (each named workload has its own).
    """
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    g = Hq // Hkv
    rng = np.random.default_rng([int(seed), int(stream)])
    Q = f32_to_bf16_bits(rng.standard_normal((B, Hq, L, D), dtype=np.float32))
    K = f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D), dtype=np.float32))
    V = f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D), dtype=np.float32))

    t = min(max(W, 1), L)                 # tail length used for the planted direction
    n_plant = min(L - 1, int(np.floor(plant * L + 0.5)))
    planted = []
    for b in range(B):
        for j in range(Hkv):
            tail = bf16_bits_to_f32(Q[b, j * g:(j + 1) * g, L - t:L, :]).astype(np.float64)
            u = tail.sum(axis=(0, 1))
            nrm = np.sqrt(np.dot(u, u))
            u = u / nrm if nrm > 0 else np.zeros(D)
            pos = np.concatenate([[0], rng.choice(np.arange(1, L), n_plant, replace=False)]) \
                if L > 1 else np.array([0])
            pos = np.sort(pos.astype(np.int64))
            rows = bf16_bits_to_f32(K[b, j, pos, :]).astype(np.float64) + 4.0 * u[None, :]
            K[b, j, pos, :] = f32_to_bf16_bits(rows.astype(np.float32))
            planted.append(pos)
    for c in outliers:
        if c < D:
            col = bf16_bits_to_f32(K[..., c]) * np.float32(10.0)
            K[..., c] = f32_to_bf16_bits(col)
    return dict(Q=Q, K=K, V=V, planted=planted)


def shared_direction(seed: int, B: int, Hq: int, Hkv: int, L: int, D: int, W: int,
                     plant: float, alpha: float = 7.0, beta: float = 4.0,
                     outliers=OUTLIER_CHANNELS, **_unused):
    """Inputs whose vertical lines come from the attention itself, to judge
    how well a selector finds them: every query of KV group j carries beta *
    e_j (a random unit direction per KV head) on top of N(0, 1), and the
    planted keys (position 0 plus a fraction of random positions) carry
    alpha * e_j, so each planted key gets a logit boost of about
    alpha * beta / sqrt(D) from every query, not only from the tail.  V ~
    N(0, 1); the outlier K channels are scaled by 10 as in ``generate``.
    Returns the same fields as ``generate``."""
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    g = Hq // Hkv
    rng = np.random.default_rng([int(seed), 1000 + int(L)])
    Qf = rng.standard_normal((B, Hq, L, D), dtype=np.float32)
    Kf = rng.standard_normal((B, Hkv, L, D), dtype=np.float32)
    V = f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D), dtype=np.float32))
    n_plant = min(L - 1, int(np.floor(plant * L + 0.5)))
    planted = []
    for b in range(B):
        for j in range(Hkv):
            e = rng.standard_normal(D)
            e = (e / np.sqrt(np.dot(e, e))).astype(np.float32)
            Qf[b, j * g:(j + 1) * g] += np.float32(beta) * e
            pos = np.concatenate([[0], rng.choice(np.arange(1, L), n_plant, replace=False)]) \
                if L > 1 else np.array([0])
            pos = np.sort(pos.astype(np.int64))
            Kf[b, j, pos, :] += np.float32(alpha) * e
            planted.append(pos)
    for c in outliers:
        if c < D:
            Kf[..., c] *= np.float32(10.0)
    return dict(Q=f32_to_bf16_bits(Qf), K=f32_to_bf16_bits(Kf), V=V, planted=planted)


def workload(name: str, **overrides) -> dict:
    """Parameters of a named workload (without its generator stream)."""
    cfg = {k: v for k, v in WORKLOADS[name].items() if k != "stream"}
    cfg.update(overrides)
    return cfg


def generate_workload(name: str, seed: int = 0, **overrides):
    """Inputs for one of the named workloads (``overrides`` may change the
    budget or bit-width of the batch-4 sweep; the drawn tensors do not depend
    on them)."""
    cfg = workload(name, **overrides)
    data = generate(seed, WORKLOADS[name]["stream"], **cfg)
    data["cfg"] = cfg
    return data


# bf16 bit patterns of the small integers the tie inputs use
_BF16_POS_ZERO, _BF16_NEG_ZERO = np.uint16(0x0000), np.uint16(0x8000)
_BF16_ONE, _BF16_MINUS_ONE = np.uint16(0x3F80), np.uint16(0xBF80)

TIE_KINDS = ("positive", "signed_zero", "all_equal")


def tie_inputs(seed: int, B: int, Hq: int, Hkv: int, L: int, W: int, k: int, kind: str,
               D: int = 128):
    """Integer-valued bf16 inputs whose selection scores tie at the k-th
    largest value, spread over the whole prefix [0, P), P = L - W.

    Q entries are drawn from {-1, 0, +1}, so the summed tail queries of a
    KV head are an integer vector c (computed here in int64 to build K; the
    tested paths compute it in float32, where it is exact).  Each prefix key
    row is one of a few patterns whose scores against c are known exactly:
      top    sign(c)                      score sum |c_d|
      mid    sign(c) on channels < D/2    score sum_{d < D/2} |c_d| (< top)
      +0     all +0.0                     score +0
      -0     -0.0 where c_d >= 0, +0.0 where c_d < 0 (every product -0)
                                          score -0
      neg    -sign(c)                     score -sum |c_d|
    kind = "positive": k // 3 top rows, 8k mid rows (the k-th largest is the
    mid score: many more ties than the rows still to take), the rest +0, -0
    and neg rows.  kind = "signed_zero": k // 2 top rows, 4k zero rows (+0 and
    -0 alternating by draw), the rest neg (the threshold is zero).
    kind = "all_equal": every tail query row is 0, so every score is a zero.
    Window rows and V are standard-normal bf16.  Returns dict(Q, K, V)."""
    if kind not in TIE_KINDS:
        raise ValueError(f"kind must be one of {TIE_KINDS}")
    g = Hq // Hkv
    P = max(0, L - W)
    t = min(max(W, 1), L)
    rng = np.random.default_rng([int(seed), 7000 + TIE_KINDS.index(kind)])
    pick = rng.integers(-1, 2, size=(B, Hq, L, D))
    Q = np.where(pick > 0, _BF16_ONE, np.where(pick < 0, _BF16_MINUS_ONE, _BF16_POS_ZERO))
    Q = Q.astype(np.uint16)
    if kind == "all_equal":
        Q[:, :, L - t:, :] = _BF16_POS_ZERO
    K = f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D), dtype=np.float32))
    V = f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, D), dtype=np.float32))
    for b in range(B):
        for j in range(Hkv):
            c = pick[b, j * g:(j + 1) * g, L - t:, :].sum(axis=(0, 1)) if kind != "all_equal" \
                else np.zeros(D, dtype=np.int64)
            top = np.where(c > 0, _BF16_ONE, np.where(c < 0, _BF16_MINUS_ONE, _BF16_POS_ZERO))
            mid = top.copy()
            mid[D // 2:] = _BF16_POS_ZERO
            neg = np.where(c > 0, _BF16_MINUS_ONE, np.where(c < 0, _BF16_ONE, _BF16_POS_ZERO))
            pz = np.full(D, _BF16_POS_ZERO, dtype=np.uint16)
            nz = np.where(c >= 0, _BF16_NEG_ZERO, _BF16_POS_ZERO)
            pats = np.stack([top, mid, pz, nz, neg]).astype(np.uint16)
            order = rng.permutation(P)
            which = np.empty(P, dtype=np.int64)
            if kind == "positive":
                n_top, n_mid = min(P, k // 3), min(P - min(P, k // 3), 8 * k)
                which[order[:n_top]] = 0
                which[order[n_top:n_top + n_mid]] = 1
                which[order[n_top + n_mid:]] = rng.choice([2, 3, 4], size=P - n_top - n_mid)
            elif kind == "signed_zero":
                n_top, n_zero = min(P, k // 2), min(P - min(P, k // 2), 4 * k)
                which[order[:n_top]] = 0
                which[order[n_top:n_top + n_zero]] = rng.choice([2, 3], size=n_zero)
                which[order[n_top + n_zero:]] = 4
            else:
                which[:] = rng.choice([2, 3], size=P)
            K[b, j, :P, :] = pats[which]
    return dict(Q=Q, K=K, V=V)
