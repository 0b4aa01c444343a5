"""The C ABI without a GPU: the library loads, exports every function the
header declares, computes sizes with the oracle's formulas, and rejects bad
arguments before enqueuing anything."""
import ctypes
import os
import re

import pytest

import paper_2608_27875_amd as hyq
from oracle import hyq_oracle as orc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(hyq.LIB_PATH):
        from paper_2608_27875_amd import build
        build.build()
    return hyq.lib()


def header_functions():
    text = open(os.path.join(ROOT, "include", "hyq.h")).read()
    return re.findall(r"^HYQ_API\s+[\w\s\*]+?\b(hyq_\w+)\s*\(", text, flags=re.M)


def test_header_symbols_exported(lib):
    names = header_functions()
    assert set(names) == set(hyq.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def shape(**kw):
    base = dict(B=1, Hq=32, Hkv=8, L=32768, D=128, window=256, budget_ppm=10000, bits_kv=8, block=64)
    base.update(kw)
    return hyq.Shape(**base)


@pytest.mark.parametrize("L,W,ppm,bits", [
    (1024, 64, 20000, 8), (8192, 128, 20000, 8), (32768, 256, 10000, 8),
    (131072, 512, 5000, 8), (16384, 256, 5000, 4), (16384, 256, 50000, 4),
    (100, 10, 1000000, 8), (100, 100, 50000, 8), (100, 10, 0, 8), (77, 0, 0, 8), (1, 0, 0, 16),
    (1, 1, 500000, 8),
])
def test_sizes_match_oracle(lib, L, W, ppm, bits):
    s = shape(B=2, Hq=40, Hkv=8, L=L, window=W, budget_ppm=ppm, bits_kv=bits)
    z = hyq.hyq_sizes_for(s)
    o = orc.sizes(L, W, ppm)
    for key in ("P", "k", "nQ", "n_qblk", "n_kvblk"):
        assert z[key] == o[key], key
    slots = o["n_kvblk"] * 64
    assert z["idx_bytes"] == 2 * 8 * o["k"] * 4
    if bits != 16:
        assert z["kq_pos_bytes"] == 2 * 8 * slots * 4
        assert z["q_codes_bytes"] == 2 * 40 * L * 128
        assert z["k_codes_bytes"] == 2 * 8 * slots * (128 if bits == 8 else 64)
        assert z["v_codes_bytes"] == 2 * 8 * o["n_kvblk"] * 128 * (64 if bits == 8 else 32)
        assert z["kv_scale_bytes"] == 2 * 8 * o["n_kvblk"] * 4
    else:
        assert z["q_codes_bytes"] == 0 and z["k_codes_bytes"] == 0


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), hyq.HYQ_EINVAL), (dict(L=0), hyq.HYQ_EINVAL), (dict(Hq=30), hyq.HYQ_EINVAL),
    (dict(window=-1), hyq.HYQ_EINVAL), (dict(budget_ppm=-5), hyq.HYQ_EINVAL),
    (dict(budget_ppm=1000001), hyq.HYQ_EINVAL), (dict(window=0), hyq.HYQ_EINVAL),
    (dict(block=0), hyq.HYQ_EINVAL),
    (dict(D=64), hyq.HYQ_EUNSUPPORTED), (dict(bits_kv=5), hyq.HYQ_EUNSUPPORTED),
    (dict(block=32), hyq.HYQ_EUNSUPPORTED), (dict(Hq=72, Hkv=8), hyq.HYQ_EUNSUPPORTED),
    (dict(kv_format=2), hyq.HYQ_EINVAL), (dict(kv_format=-1), hyq.HYQ_EINVAL),
    (dict(kv_format=hyq.FMT_FP8, bits_kv=4), hyq.HYQ_EINVAL),
])
def test_bad_shapes_rejected(lib, kw, code):
    with pytest.raises(hyq.HyqError) as e:
        hyq.hyq_sizes_for(shape(**kw))
    assert e.value.code == code
    assert hyq.hyq_last_error()


def test_null_pointers_and_args_rejected_before_launch(lib):
    """Valid shape, missing buffers: every entry point returns EINVAL without
    touching the device (none exists here)."""
    s = ctypes.byref(shape().c())
    z = hyq.hyq_sizes_for(shape())
    N = None
    assert lib.hyq_select_vertical(s, N, N, N, N, N, 0, N) == hyq.HYQ_EINVAL
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first
    assert lib.hyq_select_vertical(s, fake, fake, fake, N, fake, z["select_ws_bytes"] - 1, N) == hyq.HYQ_EINVAL
    assert "workspace" in hyq.hyq_last_error()
    assert lib.hyq_quantize(s, *([N] * 12)) == hyq.HYQ_EINVAL
    assert lib.hyq_quantize(s, fake, fake, fake, N, fake, fake, fake, fake, fake, fake, fake, N) == hyq.HYQ_EINVAL
    args = [fake] * 11
    assert lib.hyq_attn_prefill(s, *args, ctypes.c_float(0.088), fake, 2, N) == hyq.HYQ_EINVAL
    assert lib.hyq_attn_prefill(s, *args, ctypes.c_float(0.0), fake, 0, N) == hyq.HYQ_EINVAL
    assert lib.hyq_attn_prefill(s, *args, ctypes.c_float(0.088), N, 0, N) == hyq.HYQ_EINVAL
    bad = ctypes.byref(shape(D=96).c())
    assert lib.hyq_attn_prefill(bad, *args, ctypes.c_float(0.1), fake, 0, N) == hyq.HYQ_EUNSUPPORTED


def test_select_with_zero_budget_is_noop(lib):
    # k = 0: nothing to do, no pointer is needed, nothing is enqueued
    s = ctypes.byref(shape(budget_ppm=0).c())
    assert lib.hyq_select_vertical(s, None, None, None, None, None, 0, None) == hyq.HYQ_OK
    s16 = ctypes.byref(shape(bits_kv=16).c())
    assert lib.hyq_quantize(s16, *([None] * 12)) == hyq.HYQ_OK


def test_strerror(lib):
    assert hyq.hyq_strerror(0) == "success"
    assert hyq.hyq_strerror(-1) == "invalid argument"
    assert hyq.hyq_strerror(-2) == "unsupported configuration"
    assert hyq.hyq_strerror(-3) == "HIP runtime error"
