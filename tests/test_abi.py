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
    (dict(kv_format=3), hyq.HYQ_EINVAL), (dict(kv_format=-1), hyq.HYQ_EINVAL),
    (dict(kv_format=hyq.FMT_FP8, bits_kv=4), hyq.HYQ_EINVAL),
    (dict(kv_format=hyq.FMT_FP4, bits_kv=8), hyq.HYQ_EINVAL),
    (dict(window_mode=2), hyq.HYQ_EINVAL), (dict(window_mode=-1), hyq.HYQ_EINVAL),
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


def test_prefill_validates_all_three_stages_before_launch(lib):
    """hyq_prefill checks the arguments of selection, quantization and
    attention before it launches anything (no device exists here): a bad
    argument of any stage returns EINVAL."""
    s = ctypes.byref(shape().c())
    z = hyq.hyq_sizes_for(shape())
    N = None
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first
    ok_ws = ctypes.c_size_t(z["select_ws_bytes"])
    args = [fake] * 11
    # selection: workspace one byte short
    assert lib.hyq_prefill(s, *args, ctypes.c_float(0.088), fake, 0, fake,
                           ctypes.c_size_t(z["select_ws_bytes"] - 1), N) == hyq.HYQ_EINVAL
    assert "workspace" in hyq.hyq_last_error()
    # quantization: no kq_pos
    qa = [fake] * 10 + [N]
    assert lib.hyq_prefill(s, *qa, ctypes.c_float(0.088), fake, 0, fake, ok_ws, N) == hyq.HYQ_EINVAL
    # attention: bad output dtype, non-positive scale, missing output
    assert lib.hyq_prefill(s, *args, ctypes.c_float(0.088), fake, 2, fake, ok_ws, N) == hyq.HYQ_EINVAL
    assert lib.hyq_prefill(s, *args, ctypes.c_float(0.0), fake, 0, fake, ok_ws, N) == hyq.HYQ_EINVAL
    assert lib.hyq_prefill(s, *args, ctypes.c_float(0.088), N, 0, fake, ok_ws, N) == hyq.HYQ_EINVAL
    bad = ctypes.byref(shape(D=96).c())
    assert lib.hyq_prefill(bad, *args, ctypes.c_float(0.1), fake, 0, fake, ok_ws, N) == \
        hyq.HYQ_EUNSUPPORTED


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


# ---- decode cache (Algorithms 3 and 4) --------------------------------------

def _dshape(**kw):
    base = dict(B=1, Hq=32, Hkv=8, L=32768, D=128, window=128, budget_ppm=50000, bits_kv=4,
                block=64)
    base.update(kw)
    return hyq.Shape(**base)


def test_shape_struct_layout_matches_header(tmp_path):
    import subprocess
    names = [n for n, _ in hyq._Shape._fields_]
    src = ['#include <stdio.h>', '#include <stddef.h>', '#include "hyq.h"', 'int main(void) {',
           'printf("%zu\\n", sizeof(hyq_shape));']
    src += [f'printf("%zu\\n", offsetof(hyq_shape, {n}));' for n in names]
    src += ['printf("%d %d %d %d %d\\n", HYQ_WIN_FIXED, HYQ_WIN_BAND, HYQ_FMT_INT, HYQ_FMT_FP8, HYQ_FMT_FP4);',
            'return 0; }']
    c = tmp_path / "shape.c"
    c.write_text("\n".join(src))
    exe = tmp_path / "shape"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(c), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()
    assert int(out[0]) == ctypes.sizeof(hyq._Shape)
    assert [int(v) for v in out[1:1 + len(names)]] == [getattr(hyq._Shape, n).offset for n in names]
    assert [int(v) for v in out[1 + len(names):]] == [hyq.WIN_FIXED, hyq.WIN_BAND, hyq.FMT_INT,
                                                       hyq.FMT_FP8, hyq.FMT_FP4]


def test_dcache_struct_layout_matches_header(tmp_path):
    """sizeof/offsetof of hyq_dcache and hyq_dcache_sizes from the C header
    (compiled with gcc) against the binding's ctypes structures."""
    import subprocess
    fields = hyq._DCACHE_INTS + ("t",) + hyq._DCACHE_PTRS
    src = ['#include <stdio.h>', '#include <stddef.h>', '#include "hyq.h"', 'int main(void) {',
           'printf("%zu %zu\\n", sizeof(hyq_dcache), sizeof(hyq_dcache_sizes));']
    src += [f'printf("%zu\\n", offsetof(hyq_dcache, {f}));' for f in fields]
    src += [f'printf("%zu\\n", offsetof(hyq_dcache_sizes, {f}));' for f in hyq._DSIZES]
    src += ['return 0; }']
    c = tmp_path / "layout.c"
    c.write_text("\n".join(src))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(c), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()
    vals = [int(v) for v in out]
    assert vals[0] == ctypes.sizeof(hyq._DCache) and vals[1] == ctypes.sizeof(hyq._DCacheSizes)
    offs = vals[2:2 + len(fields)]
    assert offs == [getattr(hyq._DCache, f).offset for f in fields]
    assert vals[2 + len(fields):] == [getattr(hyq._DCacheSizes, f).offset for f in hyq._DSIZES]


@pytest.mark.parametrize("L,W,ppm,bits,extra,ws", [
    (32768, 128, 50000, 4, 1024, 0), (1000, 64, 20000, 8, 0, 0), (517, 100, 20000, 4, 200, 0),
    (200, 64, 1000000, 4, 64, 0), (64, 64, 50000, 8, 140, 0), (450, 96, 0, 8, 1, 0),
    (32768, 128, 50000, 4, 1024, 128), (700, 200, 30000, 8, 300, 192),
])
def test_dcache_geometry(lib, L, W, ppm, bits, extra, ws):
    s = _dshape(L=L, window=W, budget_ppm=ppm, bits_kv=bits, staging=ws)
    c, z = hyq.hyq_dcache_init(s, L + extra)
    o = orc.sizes(L, W, ppm)
    rup = lambda x: -(-x // 64) * 64
    Ws = ws or hyq.DECODE_WS
    assert c.n_vl == o["k"] and c.n_frozen == o["nQ"] and c.staging == Ws
    assert c.vl_rows == rup(o["k"]) and c.ring_rows == rup(W) + Ws
    assert c.cap_blocks == o["n_kvblk"] + -(-extra // 64)
    assert (c.n_merged, c.ring_head, c.n_staged, c.t) == (0, 0, 0, L)
    BH, nfp, cap = 8, c.vl_rows + c.ring_rows, c.cap_blocks
    assert z["k_codes_bytes"] == BH * cap * 64 * (128 if bits == 8 else 64)
    assert z["v_codes_bytes"] == BH * cap * 128 * (64 if bits == 8 else 32)
    assert z["fp_k_bytes"] == z["fp_v_bytes"] == BH * nfp * 128 * 2
    assert z["q_pos_bytes"] == BH * cap * 64 * 4 and z["vl_pos_bytes"] == BH * o["k"] * 4
    assert z["freeze_ws_bytes"] == hyq.hyq_sizes_for(s)["select_ws_bytes"]
    assert z["attn_ws_bytes"] > 0


@pytest.mark.parametrize("kw,max_extra", [
    (dict(window=32), 0), (dict(L=100, window=128), 0), (dict(bits_kv=16), 0),
    (dict(), -1), (dict(D=64), 0), (dict(staging=32), 0), (dict(staging=100), 0),
    (dict(window=128, staging=192), 0), (dict(staging=-64), 0),
])
def test_dcache_bad_geometry_rejected(lib, kw, max_extra):
    s = _dshape(**kw)
    with pytest.raises(hyq.HyqError):
        hyq.hyq_dcache_init(s, s.L + max_extra)


def test_dcache_rejects_fp6_query_format(lib):
    """HYQ_FMT_FP4Q6 only sets the prefill's query codes; a decode cache with it is refused."""
    s = _dshape(bits_kv=4, kv_format=hyq.FMT_FP4Q6)
    with pytest.raises(hyq.HyqError) as e:
        hyq.hyq_dcache_init(s, s.L)
    assert e.value.code in (hyq.HYQ_EUNSUPPORTED, hyq.HYQ_EINVAL)
    hyq.hyq_dcache_init(_dshape(bits_kv=4, kv_format=hyq.FMT_FP4), s.L)   # FP4 caches are fine


def test_decode_calls_reject_bad_arguments_before_launch(lib):
    s = _dshape(L=1000, window=64, budget_ppm=20000, bits_kv=8)
    c, z = hyq.hyq_dcache_init(s, 1200)
    fake = 0x1000                      # never dereferenced: validation fails first
    N = None
    # buffers missing
    assert lib.hyq_decode_append(ctypes.byref(c), ctypes.c_void_p(fake), ctypes.c_void_p(fake),
                                 N) == hyq.HYQ_EINVAL
    for n in hyq._DCACHE_PTRS:
        setattr(c, n, fake)
    f = ctypes.c_void_p(fake)
    # bad state
    c.n_staged = 65
    assert lib.hyq_decode_append(ctypes.byref(c), f, f, N) == hyq.HYQ_EINVAL
    c.n_staged = 0
    c.ring_head = 5
    assert lib.hyq_decode_attn(ctypes.byref(c), f, ctypes.c_float(0.088), f, 0, f,
                               z["attn_ws_bytes"], N) == hyq.HYQ_EINVAL
    c.ring_head = 0
    # full cache: a merge is due and every block is in use
    c.n_staged = 64
    c.n_merged = c.cap_blocks - -(-c.n_frozen // 64)
    assert lib.hyq_decode_append(ctypes.byref(c), f, f, N) == hyq.HYQ_EINVAL
    assert "full" in hyq.hyq_last_error()
    assert c.n_staged == 64                        # state unchanged
    c.n_merged = 0
    # workspace too small, bad out dtype, bad scale, missing q
    assert lib.hyq_decode_attn(ctypes.byref(c), f, ctypes.c_float(0.088), f, 0, f,
                               z["attn_ws_bytes"] - 1, N) == hyq.HYQ_EINVAL
    assert "workspace" in hyq.hyq_last_error()
    assert lib.hyq_decode_attn(ctypes.byref(c), f, ctypes.c_float(0.088), f, 2, f,
                               z["attn_ws_bytes"], N) == hyq.HYQ_EINVAL
    assert lib.hyq_decode_attn(ctypes.byref(c), f, ctypes.c_float(-1.0), f, 0, f,
                               z["attn_ws_bytes"], N) == hyq.HYQ_EINVAL
    assert lib.hyq_decode_attn(ctypes.byref(c), N, ctypes.c_float(0.088), f, 0, f,
                               z["attn_ws_bytes"], N) == hyq.HYQ_EINVAL
    # freeze: shape that does not match the cache
    other = ctypes.byref(_dshape(L=1001, window=64, budget_ppm=20000, bits_kv=8).c())
    assert lib.hyq_freeze(other, f, f, f, ctypes.byref(c), f, z["freeze_ws_bytes"],
                          N) == hyq.HYQ_EINVAL
    assert "match" in hyq.hyq_last_error()
    assert lib.hyq_freeze(ctypes.byref(s.c()), f, f, f, ctypes.byref(c), f,
                          z["freeze_ws_bytes"] - 1, N) == hyq.HYQ_EINVAL


def test_decode_attn_noalloc_rejects_before_launch(lib):
    """The allocation-free decode call validates like hyq_decode_attn and
    refuses a launch whose partials exceed its scratch, before any HIP call."""
    fake = 0x1000
    f = ctypes.c_void_p(fake)
    N = None
    s = _dshape(L=1000, window=64, budget_ppm=20000, bits_kv=8)
    c, _ = hyq.hyq_dcache_init(s, 1200)
    for n in hyq._DCACHE_PTRS:
        setattr(c, n, fake)
    assert lib.hyq_decode_attn_noalloc(ctypes.byref(c), f, ctypes.c_float(0.088), f, 2,
                                       N) == hyq.HYQ_EINVAL
    assert lib.hyq_decode_attn_noalloc(ctypes.byref(c), N, ctypes.c_float(0.088), f, 0,
                                       N) == hyq.HYQ_EINVAL
    big = _dshape(B=64, Hq=32, Hkv=8, L=32768, window=128, budget_ppm=50000, bits_kv=4)
    cb, _ = hyq.hyq_dcache_init(big, 32768 + 64)
    for n in hyq._DCACHE_PTRS:
        setattr(cb, n, fake)
    assert lib.hyq_decode_attn_noalloc(ctypes.byref(cb), f, ctypes.c_float(0.088), f, 0,
                                       N) == hyq.HYQ_EUNSUPPORTED
    assert "scratch" in hyq.hyq_last_error()
