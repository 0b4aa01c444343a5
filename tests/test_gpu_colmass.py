"""GPU parity of the exact column-mass selector (eq. vl_score, eq. vl_topk):
the column mass itself within a relative 1e-5 of the oracle's float64 value
(the GPU sums in float32, in another order), the selected positions equal to
the oracle's (the planted vertical lines keep the k-th score clear of its
neighbours; a tie-robust validity check is applied as well), then the rest of
the prefill and the decode Freeze on those positions, as for Algorithm 1."""
import dataclasses
import zlib

import numpy as np
import pytest

import gpu_common as gc
import paper_2608_27875_amd as hyq
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen

pytestmark = pytest.mark.gpu

COL = hyq.SEL_COLMASS
REL = 1e-5


def valid_topk(S, sel, k, rel):
    """sel is a top-k set of S up to a relative tolerance: every chosen score
    is >= the k-th largest minus rel * max, every other one <= it plus that."""
    kth = np.sort(S)[::-1][k - 1]
    tol = rel * S.max()
    chosen = np.zeros(len(S), bool)
    chosen[sel] = True
    return len(set(sel.tolist())) == k and np.all(S[chosen] >= kth - tol) and \
        np.all(S[~chosen] <= kth + tol)


def check_colmass(shape, d, g):
    idx, S = orc.select_vertical_colmass(d["Q"], d["K"], shape.Hkv, shape.window,
                                         shape.budget_ppm)
    z = g["sizes"]
    gs = g["scores"].reshape(S.shape)
    err = np.abs(gs - S) / S.max(axis=-1, keepdims=True)
    print(f"  column mass: max rel err {err.max():.2e}", flush=True)
    assert err.max() <= REL
    gidx = g["idx"].reshape(idx.shape)
    for ix in np.ndindex(*idx.shape[:-1]):
        assert valid_topk(S[ix], gidx[ix], z["k"], 2 * REL), ix
    np.testing.assert_array_equal(gidx, idx)
    return idx


# (name, B, Hq, Hkv, L, W, budget_ppm, bits)
SMALL = [
    ("cm_cfg1", 1, 1, 1, 1024, 64, 20000, 8),
    ("cm_gqa4_ragged", 1, 8, 2, 1000, 64, 20000, 8),
    ("cm_w100_t_ragged", 1, 8, 2, 777, 100, 30000, 4),
    ("cm_b2_g5", 2, 10, 2, 600, 48, 30000, 8),
    ("cm_w_over_l", 1, 4, 1, 90, 200, 0, 8),
    ("cm_tiny", 1, 2, 1, 40, 8, 100000, 8),
]


def _inputs(name, B, Hq, Hkv, L, W):
    return gen.generate(0, zlib.crc32(name.encode()) % 10007 + 40000, B=B, Hq=Hq, Hkv=Hkv, L=L,
                        D=128, W=max(W, 1), plant=0.02)


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_colmass_small_full_path(case):
    name, B, Hq, Hkv, L, W, ppm, bits = case
    print(f"case {name}", flush=True)
    d = _inputs(name, B, Hq, Hkv, L, W)
    shape = hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=L, window=W, budget_ppm=ppm, bits_kv=bits,
                      selector=COL)
    g = gc.run_gpu(shape, d)
    if g["sizes"]["k"] == 0:
        assert g["scores"] is None
        return
    idx = check_colmass(shape, d, g)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, bits)
    c = gc.canonical(shape, g)
    for key in ("kq_pos", "q_codes", "k_codes", "v_codes"):
        np.testing.assert_array_equal(c[key], qz[key], err_msg=key)
    O = orc.attention(d["Q"], d["K"], d["V"], W, bits, idx, qz)
    mx, mean = gc.attention_error(g["out"].reshape(O.shape), O)
    print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN


@pytest.mark.timeout(300)
def test_colmass_32k():
    """The 32k GQA workload selected by column mass (the 256 tail queries of
    each of the 32 heads against 32k keys): scores and positions in full,
    attention on 4 heads x 256 rows."""
    shape = dataclasses.replace(gc.shape_of(gen.workload(gen.GQA_32K)), selector=COL)
    print("32k colmass: generating", flush=True)
    d = gen.generate_workload(gen.GQA_32K, seed=0)
    g = gc.run_gpu(shape, d, keep_out_on_gpu=True)
    print("  oracle column mass", flush=True)
    idx = check_colmass(shape, d, g)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, shape.window, 8)
    rng = np.random.default_rng(35)
    heads = [(0, h) for h in sorted(rng.choice(shape.Hq, size=4, replace=False))]
    rows = gc.sample_rows(shape.L, shape.window, 256, 35)
    O = orc.attention(d["Q"], d["K"], d["V"], shape.window, 8, idx, qz, heads=heads, rows=rows)
    import torch
    out = g["out_dev"]
    rt = torch.from_numpy(rows).to(out.device)
    Og = np.stack([out[b, h].index_select(0, rt).cpu().numpy() for b, h in heads])
    mx, mean = gc.attention_error(Og, O)
    print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN


def test_colmass_freeze():
    """Freeze (Algorithm 4) with the column-mass selector: vertical positions
    and every cached block as the oracle's Freeze with the same selector."""
    import test_gpu_decode as td
    N, W = 700, 64
    shape = hyq.Shape(B=1, Hq=8, Hkv=2, L=N, window=W, budget_ppm=50000, bits_kv=4, selector=COL)
    d = _inputs("cm_freeze", 1, 8, 2, N, W)
    cache = hyq.DecodeCache(shape, N + 100, "cuda")
    Q, K, V = (gc.to_dev(d[n]) for n in ("Q", "K", "V"))
    hyq.hyq_freeze(shape, Q, K, V, cache)
    oc = orc.freeze(d["Q"], d["K"], d["V"], 2, W, 50000, 4, selector="colmass")
    oc["vl_pos"] = np.asarray(oc["vl_pos"])
    td.check_cache(cache, oc)
    td.check_attention(cache, oc, np.random.default_rng(3), label="colmass freeze")


@pytest.mark.timeout(600)
def test_colmass_batch4_16k():
    """The batch-4, 40q/8kv, 16k workload (2% budget) selected by column
    mass: every batch and KV head's scores and positions in full, attention
    on 2 heads x 256 rows of the last batch entry."""
    shape = dataclasses.replace(gc.shape_of(gen.workload(gen.BATCH4_16K, budget_ppm=20000, bits=8)),
                                selector=COL)
    print("batch-4 16k colmass: generating", flush=True)
    d = gen.generate_workload(gen.BATCH4_16K, seed=0)
    g = gc.run_gpu(shape, d, keep_out_on_gpu=True)
    print("  oracle column mass", flush=True)
    idx = check_colmass(shape, d, g)
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, shape.window, 8)
    rng = np.random.default_rng(55)
    heads = [(shape.B - 1, h) for h in sorted(rng.choice(shape.Hq, size=2, replace=False))]
    rows = gc.sample_rows(shape.L, shape.window, 256, 55)
    O = orc.attention(d["Q"], d["K"], d["V"], shape.window, 8, idx, qz, heads=heads, rows=rows)
    import torch
    out = g["out_dev"]
    rt = torch.from_numpy(rows).to(out.device)
    Og = np.stack([out[b, h].index_select(0, rt).cpu().numpy() for b, h in heads])
    mx, mean = gc.attention_error(Og, O)
    print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN


def test_shared_direction_both_selectors():
    """Vertical lines made by the attention itself (gen.shared_direction): both
    GPU selectors give the oracle's positions (Algorithm 1 bit for bit, its
    scores too; the column mass within REL), and both find most planted
    lines."""
    B, Hq, Hkv, L, W, ppm = 1, 8, 2, 8192, 128, 20000
    print("case shared_direction 8k", flush=True)
    d = gen.shared_direction(0, B=B, Hq=Hq, Hkv=Hkv, L=L, D=128, W=W, plant=0.01)
    base = hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=L, window=W, budget_ppm=ppm, bits_kv=8)
    g1 = gc.run_gpu(base, d)
    idx1, _ = gc.check_select_quant(base, d, g1)
    shape = dataclasses.replace(base, selector=COL)
    g2 = gc.run_gpu(shape, d)
    idx2 = check_colmass(shape, d, g2)
    z = g1["sizes"]
    for name, idx in (("tail proxy", idx1), ("column mass", idx2)):
        rec = []
        for bj, pos in enumerate(d["planted"]):
            pp = set(p for p in pos.tolist() if p < z["P"])
            rec.append(len(pp & set(idx.reshape(-1, z["k"])[bj].tolist())) / min(len(pp), z["k"]))
        print(f"  {name} recall {np.mean(rec):.3f}", flush=True)
        assert np.mean(rec) >= 0.7
