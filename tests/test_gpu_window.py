"""GPU parity of the window readings: the per-query window of eq. (win_def)
(HYQ_WIN_BAND) against the oracle's band mode, and the rows of the final
query chunk against Algorithm 2's Stage 3 taken literally (segments A and B
unmasked, C causal).  Selection and quantization are the fixed-window ones in
both modes (compared bit-exact); attention within max-abs 2e-3, mean-abs 2e-4."""
import dataclasses
import zlib

import numpy as np
import pytest

import gpu_common as gc
import paper_2608_27875_amd as hyq
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen

pytestmark = pytest.mark.gpu

BAND = hyq.WIN_BAND

# (name, B, Hq, Hkv, L, W, budget_ppm, bits, fmt)
SMALL = [
    ("band_cfg1", 1, 1, 1, 1024, 64, 20000, 8, hyq.FMT_INT),
    ("band_gqa4_ragged", 1, 8, 2, 1000, 64, 20000, 8, hyq.FMT_INT),
    ("band_w100", 1, 8, 2, 777, 100, 30000, 8, hyq.FMT_INT),
    ("band_int4_b2", 2, 4, 2, 640, 96, 50000, 4, hyq.FMT_INT),
    ("band_fp8_g5", 1, 10, 2, 600, 48, 30000, 8, hyq.FMT_FP8),
    ("band_g8_int4", 1, 16, 2, 500, 128, 20000, 4, hyq.FMT_INT),
    ("band_budget0", 1, 4, 1, 700, 200, 0, 8, hyq.FMT_INT),
    ("band_all_prefix_vertical", 1, 4, 1, 300, 40, 1000000, 8, hyq.FMT_INT),
    ("band_w_covers_all", 1, 4, 1, 200, 256, 50000, 8, hyq.FMT_INT),
    ("band_tiny", 1, 2, 1, 17, 4, 100000, 8, hyq.FMT_INT),
    ("band_bits16", 1, 4, 1, 300, 64, 20000, 16, hyq.FMT_INT),
]


def _inputs(name, B, Hq, Hkv, L, W, seed=0):
    return gen.generate(seed, zlib.crc32(name.encode()) % 10007 + 30000, B=B, Hq=Hq, Hkv=Hkv, L=L,
                        D=128, W=max(W, 1), plant=0.02)


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_band_small_full_parity(case):
    name, B, Hq, Hkv, L, W, ppm, bits, fmt = case
    print(f"case {name}", flush=True)
    d = _inputs(name, B, Hq, Hkv, L, W)
    shape = hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=L, window=W, budget_ppm=ppm, bits_kv=bits,
                      kv_format=fmt, window_mode=BAND)
    g = gc.run_gpu(shape, d)
    idx, qz = gc.check_select_quant(shape, d, g)
    O = orc.attention(d["Q"], d["K"], d["V"], W, bits, idx, qz if bits != 16 else None,
                      window_mode="band")
    Og = g["out"].reshape(O.shape)
    mx, mean = gc.attention_error(Og, O)
    print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN


@pytest.mark.timeout(300)
def test_band_32k():
    """The 32k GQA workload with the per-query window (4 heads x 512 rows,
    always including rows W-1, W, P-1, P and L-1)."""
    cfg = gen.workload(gen.GQA_32K)
    shape = dataclasses.replace(gc.shape_of(cfg), window_mode=BAND)
    print("32k band: generating", flush=True)
    d = gen.generate_workload(gen.GQA_32K, seed=0)
    g = gc.run_gpu(shape, d, keep_out_on_gpu=True)
    idx, qz = gc.check_select_quant(shape, d, g)
    rng = np.random.default_rng(34)
    heads = [(0, h) for h in sorted(rng.choice(shape.Hq, size=4, replace=False))]
    rows = np.union1d(gc.sample_rows(shape.L, shape.window, 512, 34),
                      [shape.window - 1, shape.window])
    O = orc.attention(d["Q"], d["K"], d["V"], shape.window, 8, idx, qz, heads=heads, rows=rows,
                      window_mode="band")
    import torch
    out = g["out_dev"]
    rt = torch.from_numpy(rows).to(out.device)
    Og = np.stack([out[b, h].index_select(0, rt).cpu().numpy() for b, h in heads])
    mx, mean = gc.attention_error(Og, O)
    print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN


@pytest.mark.parametrize("name", [gen.SMALL, gen.GQA_8K])
def test_final_chunk_matches_literal_algorithm(name):
    """The kernel's (fixed-window) rows of the final chunk [L-W, L) against
    Algorithm 2's Stage 3 taken literally (A and B unmasked, C causal,
    tile-by-tile online softmax), every head."""
    cfg = gen.workload(name)
    shape = gc.shape_of(cfg)
    d = gen.generate_workload(name, seed=0)
    g = gc.run_gpu(shape, d)
    idx, qz = gc.check_select_quant(shape, d, g)
    Oc = orc.attention_final_chunk(d["Q"], d["K"], d["V"], shape.window, shape.bits_kv, idx, qz)
    P = shape.L - shape.window
    Og = g["out"].reshape(shape.B * shape.Hq, shape.L, 128)[:, P:]
    mx, mean = gc.attention_error(Og, Oc)
    print(f"  {name} final chunk: max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN
