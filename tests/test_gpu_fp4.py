"""GPU parity for FP4 codes (OCP E2M1 keys and values with c_B = 6), with
E4M3 queries (HYQ_FMT_FP4) and with FP6 E2M3 queries (HYQ_FMT_FP4Q6, both
MFMA operands at most 6 bits): the HIP path through the C ABI against the
CPU oracle on the same seeded inputs.  Selection, partition, code bytes and
scales bit-exact; attention output within max-abs 2e-3 and mean-abs 2e-4."""
import zlib

import numpy as np
import pytest

import gpu_common as gc
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen

pytestmark = pytest.mark.gpu

FP4 = gc.hyq.FMT_FP4
FP4Q6 = gc.hyq.FMT_FP4Q6
FMTS = pytest.mark.parametrize("fmt", [FP4, FP4Q6], ids=["q8", "q6"])

# (name, B, Hq, Hkv, L, W, budget_ppm)
SMALL = [
    ("fp4_cfg1", 1, 1, 1, 1024, 64, 20000),
    ("fp4_gqa4_ragged", 1, 8, 2, 1000, 64, 20000),
    ("fp4_g5", 1, 10, 2, 600, 48, 30000),
    ("fp4_g8", 1, 16, 2, 400, 64, 20000),
    ("fp4_mha3_b2", 2, 3, 3, 333, 20, 60000),
    ("fp4_window_only", 1, 4, 1, 700, 96, 0),
    ("fp4_uniform_no_window", 1, 4, 1, 650, 0, 0),
    ("fp4_all_prefix_vertical", 1, 4, 1, 300, 40, 1000000),
    ("fp4_tiny", 1, 2, 1, 17, 4, 100000),
    ("fp4_one_token", 1, 2, 1, 1, 1, 0),
]


def _inputs(name, B, Hq, Hkv, L, W, seed=0):
    return gen.generate(seed, zlib.crc32(name.encode()) % 10007, B=B, Hq=Hq, Hkv=Hkv, L=L, D=128,
                        W=max(W, 1), plant=0.02)


def _shape(B, Hq, Hkv, L, W, ppm, window_mode=0, fmt=FP4):
    return gc.hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=L, window=W, budget_ppm=ppm, bits_kv=4,
                        kv_format=fmt, window_mode=window_mode)


def _check_small(d, shape, skip_channel=None):
    g = gc.run_gpu(shape, d)
    idx, qz = gc.check_select_quant(shape, d, g)
    mode = "band" if shape.window_mode == gc.hyq.WIN_BAND else "fixed"
    O = orc.attention(d["Q"], d["K"], d["V"], shape.window, 4, idx, qz, window_mode=mode)
    Og = g["out"].reshape(O.shape)
    if skip_channel is None:
        mx, mean = gc.attention_error(Og, O)
        print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
        assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN
    else:
        rel = gc.scaled_error(Og, O)
        keep = np.arange(O.shape[-1]) != skip_channel
        mx, mean = gc.attention_error(Og[..., keep], O[..., keep])
        print(f"  scaled max {rel:.3e}; other channels max-abs {mx:.3e} mean-abs {mean:.3e}",
              flush=True)
        assert rel <= gc.TOL_MAX and mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN
    return g


@FMTS
@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_fp4_small_full_parity(case, fmt):
    name, B, Hq, Hkv, L, W, ppm = case
    print(f"case {name} fmt {fmt}", flush=True)
    d = _inputs(name, B, Hq, Hkv, L, W)
    _check_small(d, _shape(B, Hq, Hkv, L, W, ppm, fmt=fmt))


@FMTS
def test_fp4_band_window(fmt):
    """The per-query window with FP4 codes."""
    d = _inputs("fp4_band", 1, 8, 2, 900, 96)
    _check_small(d, _shape(1, 8, 2, 900, 96, 20000, window_mode=gc.hyq.WIN_BAND, fmt=fmt))


@FMTS
def test_fp4_zeros_signs_and_saturation(fmt):
    """Blocks with exact zeros and negative zeros (E2M1 codes 0 / 8), a block
    that is all zero (scale 0), tiny entries that round to signed zero, and
    one huge outlier (its code is +-6; in V it makes one block's scale dwarf
    all others).  Outputs on the outlier channel reach ~1e3, so the bound
    there scales with the row's magnitude."""
    L, W = 520, 40
    d = _inputs("fp4_edges", 1, 4, 1, L, W)
    for name in ("Q", "K", "V"):
        x = gen.bf16_bits_to_f32(d[name])
        x[..., 3] = 0.0
        x[..., 5] = -0.0
        x[..., 64:128, :] = 0.0                        # whole zero blocks (rows 64..127)
        x[..., 130:140, 7] = 1e-6 * np.sign(x[..., 130:140, 7] + 0.5)
        x[..., 200, 9] = 3.0e4                         # one outlier in a block
        d[name] = gen.f32_to_bf16_bits(x)
    g = _check_small(d, _shape(1, 4, 1, L, W, 30000, fmt=fmt), skip_channel=9)
    nib = gc.unpack_codes4(g["k_codes"].view(np.uint8), fmt)
    assert np.any(nib == 0x8) and np.any(nib == 0x7)
    if fmt == FP4Q6:   # E2M3 query codes: -0 and +-7.5 occur
        qc = g["q_codes"].view(np.uint8)
        assert np.any(qc == 0x20) and np.any((qc & 0x1F) == 0x1F) and qc.max() <= 0x3F


@FMTS
def test_fp4_deterministic(fmt):
    d = _inputs("fp4_det", 1, 8, 2, 900, 64)
    shape = _shape(1, 8, 2, 900, 64, 20000, fmt=fmt)
    g1 = gc.run_gpu(shape, d)
    g2 = gc.run_gpu(shape, d)
    for k in ("idx", "q_codes", "k_codes", "v_codes", "kq_pos", "out"):
        np.testing.assert_array_equal(g1[k], g2[k], err_msg=k)


@FMTS
@pytest.mark.timeout(300)
def test_fp4_32k(fmt):
    """The 32k GQA workload with FP4 codes (4 heads x 512 sampled rows)."""
    cfg = gen.workload(gen.GQA_32K, bits=4, fmt=fmt)
    print("32k fp4: generating", flush=True)
    d = gen.generate_workload(gen.GQA_32K, seed=0)
    shape = gc.shape_of(cfg)
    print("  running HIP path", flush=True)
    g = gc.run_gpu(shape, d, keep_out_on_gpu=True)
    print("  oracle selection + quantization", flush=True)
    idx, qz = gc.check_select_quant(shape, d, g)
    rng = np.random.default_rng(34)
    heads = sorted(rng.choice(shape.Hq, size=4, replace=False).tolist())
    heads = [(0, h) for h in heads]
    rows = gc.sample_rows(shape.L, shape.window, 512, 34)
    print(f"  oracle attention on {len(heads)} heads x {len(rows)} rows", flush=True)
    O = orc.attention(d["Q"], d["K"], d["V"], shape.window, 4, idx, qz, heads=heads, rows=rows)
    out = g["out_dev"]
    import torch
    rt = torch.from_numpy(rows).to(out.device)
    Og = np.stack([out[b, h].index_select(0, rt).cpu().numpy() for b, h in heads])
    mx, mean = gc.attention_error(Og, O)
    print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN


@FMTS
@pytest.mark.timeout(600)
def test_fp4_128k(fmt):
    """The 131k-token workload (window 512, 0.5% budget) with FP4 codes:
    selection and every code in full, attention on 2 heads x 256 rows."""
    cfg = gen.workload(gen.GQA_128K, bits=4, fmt=fmt)
    print("128k fp4: generating", flush=True)
    d = gen.generate_workload(gen.GQA_128K, seed=0)
    shape = gc.shape_of(cfg)
    print("  running HIP path", flush=True)
    g = gc.run_gpu(shape, d, keep_out_on_gpu=True)
    print("  oracle selection + quantization", flush=True)
    idx, qz = gc.check_select_quant(shape, d, g)
    rng = np.random.default_rng(44)
    heads = [(0, h) for h in sorted(rng.choice(shape.Hq, size=2, replace=False).tolist())]
    rows = gc.sample_rows(shape.L, shape.window, 256, 44)
    print(f"  oracle attention on {len(heads)} heads x {len(rows)} rows", flush=True)
    O = orc.attention(d["Q"], d["K"], d["V"], shape.window, 4, idx, qz, heads=heads, rows=rows)
    out = g["out_dev"]
    import torch
    rt = torch.from_numpy(rows).to(out.device)
    Og = np.stack([out[b, h].index_select(0, rt).cpu().numpy() for b, h in heads])
    mx, mean = gc.attention_error(Og, O)
    print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN
