"""GPU parity of the decode path: Freeze (Algorithm 4), the staging buffer
and its merges, and decode attention (Algorithm 3), through the C ABI
against the oracle on the same seeded inputs.

Bit-exact: vertical-line positions, quantized-token positions, every code
and scale of every block (frozen and merged), the bf16 rows of the
vertical lines, the window and the staging buffer.  Attention output:
max-abs 2e-3, mean-abs 2e-4 against the oracle's float64 softmax."""
import zlib

import numpy as np
import pytest

import gpu_common as gc
import paper_2608_27875_amd as hyq
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen

pytestmark = pytest.mark.gpu


def _fmt(shape):
    return gc.fmt_name(shape)


def _rows(rng, B, H, D=128):
    return gen.f32_to_bf16_bits(rng.standard_normal((B, H, D)).astype(np.float32))


def _gpu_view(cache: hyq.DecodeCache) -> dict:
    """The cache's device buffers in the oracle's terms (codes unpacked, V
    blocks back to token-major)."""
    c = cache.c
    BH, D, cap = c.B * c.Hkv, c.D, c.cap_blocks
    b = {n: t.cpu().numpy() for n, t in cache.bufs.items() if n not in ("fp_k", "fp_v")}
    nfp = c.vl_rows + c.ring_rows
    fk = cache.bufs["fp_k"].view(__import__("torch").int16).cpu().numpy().view(np.uint16)
    fv = cache.bufs["fp_v"].view(__import__("torch").int16).cpu().numpy().view(np.uint16)
    ctype = np.int8 if c.kv_format == hyq.FMT_INT else np.uint8
    if c.bits_kv == 8:
        kc = b["k_codes"][:BH * cap * 64 * D].view(ctype).reshape(BH, cap * 64, D)
        vc = b["v_codes"][:BH * cap * D * 64].view(ctype).reshape(BH, cap, D, 64)
    else:
        kc = gc.unpack_codes4(b["k_codes"][:BH * cap * 64 * D // 2].reshape(BH, cap * 64, D // 2),
                              c.kv_format)
        vc = gc.unpack_codes4(b["v_codes"][:BH * cap * D * 32].reshape(BH, cap, D, 32), c.kv_format)
    vc = vc.transpose(0, 1, 3, 2).reshape(BH, cap * 64, D)
    return dict(kc=kc, vc=vc, ks=b["k_scale"][:BH * cap].reshape(BH, cap),
                vs=b["v_scale"][:BH * cap].reshape(BH, cap),
                q_pos=b["q_pos"][:BH * cap * 64].reshape(BH, cap * 64),
                vl_pos=b["vl_pos"][:BH * c.n_vl].reshape(BH, c.n_vl),
                fk=fk[:BH * nfp * D].reshape(BH, nfp, D), fv=fv[:BH * D * nfp].reshape(BH, D, nfp))


def check_cache(cache: hyq.DecodeCache, oc: dict):
    """Every buffer of the GPU cache against the oracle's cache."""
    c = cache.c
    g = _gpu_view(cache)
    BH, W = c.B * c.Hkv, c.window
    nbf = -(-c.n_frozen // 64)
    assert c.t == oc["t"]
    np.testing.assert_array_equal(g["vl_pos"], oc["vl_pos"].reshape(BH, -1))
    for bj in range(BH):
        nb = len(oc["k_blocks"][bj])
        assert nb == nbf + c.n_merged, (nb, nbf, c.n_merged)
        for i in range(nb):
            n = len(oc["q_pos"][bj][i])
            r = slice(i * 64, i * 64 + n)
            np.testing.assert_array_equal(g["kc"][bj, r], oc["k_blocks"][bj][i][:n],
                                          err_msg=f"k codes bj {bj} block {i}")
            np.testing.assert_array_equal(g["vc"][bj, r], oc["v_blocks"][bj][i][:n],
                                          err_msg=f"v codes bj {bj} block {i}")
            np.testing.assert_array_equal(g["q_pos"][bj, r], oc["q_pos"][bj][i])
            assert np.all(g["kc"][bj, i * 64 + n:(i + 1) * 64] == 0)
            assert np.all(g["vc"][bj, i * 64 + n:(i + 1) * 64] == 0)
            assert np.all(g["q_pos"][bj, i * 64 + n:(i + 1) * 64] == hyq.KQ_POS_PAD)
            for key, okey in (("ks", "k_scales"), ("vs", "v_scales")):
                assert np.float32(g[key][bj, i]).view(np.uint32) == \
                    np.float32(oc[okey][bj][i]).view(np.uint32), (key, bj, i)
        k = c.n_vl
        np.testing.assert_array_equal(g["fk"][bj, :k], oc["vl_k"][bj])
        np.testing.assert_array_equal(g["fv"][bj, :, :k].T, oc["vl_v"][bj])
        ring = [(c.ring_head + i) % c.ring_rows for i in range(W + c.n_staged)]
        rows = np.array(ring) + c.vl_rows
        want_k = np.stack(oc["win_k"][bj] + oc["st_k"][bj])
        want_v = np.stack(oc["win_v"][bj] + oc["st_v"][bj])
        np.testing.assert_array_equal(g["fk"][bj, rows], want_k)
        np.testing.assert_array_equal(g["fv"][bj][:, rows].T, want_v)


def check_attention(cache: hyq.DecodeCache, oc: dict, rng, out_dtype=0, label=""):
    import torch
    c = cache.c
    q = _rows(rng, c.B, c.Hq)
    out = torch.empty((c.B, c.Hq, c.D), dtype=torch.float32 if out_dtype == 0 else torch.bfloat16,
                      device="cuda")
    hyq.hyq_decode_attn(cache, gc.to_dev(q), out, out_dtype=out_dtype)
    torch.cuda.synchronize()
    O = orc.decode_attention(q, oc)
    Og = out.float().cpu().numpy()
    mx, mean = gc.attention_error(Og, O)
    print(f"  {label} t={c.t} merged={c.n_merged} staged={c.n_staged}: "
          f"max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    tol = gc.TOL_MAX + (4e-3 if out_dtype else 0.0)
    assert mx <= tol and mean <= gc.TOL_MEAN + (1e-3 if out_dtype else 0.0)
    return Og


def freeze_both(shape: hyq.Shape, d: dict, max_tokens: int):
    cache = hyq.DecodeCache(shape, max_tokens, "cuda")
    Q, K, V = (gc.to_dev(d[n]) for n in ("Q", "K", "V"))
    hyq.hyq_freeze(shape, Q, K, V, cache)
    oc = orc.freeze(d["Q"], d["K"], d["V"], shape.Hkv, shape.window, shape.budget_ppm,
                    shape.bits_kv, fmt=_fmt(shape), staging=shape.staging or hyq.DECODE_WS)
    oc["vl_pos"] = np.asarray(oc["vl_pos"])
    return cache, oc


def append_both(cache, oc, rng):
    c = cache.c
    kn, vn = _rows(rng, c.B, c.Hkv), _rows(rng, c.B, c.Hkv)
    hyq.hyq_decode_append(cache, gc.to_dev(kn), gc.to_dev(vn))
    orc.decode_append(oc, kn, vn)


# (name, B, Hq, Hkv, N, W, budget_ppm, bits, fmt)
SMALL = [
    ("int8_g4", 1, 8, 2, 700, 64, 30000, 8, hyq.FMT_INT),
    ("int4_g4", 1, 8, 2, 700, 64, 30000, 4, hyq.FMT_INT),
    ("fp8_g4", 1, 8, 2, 700, 64, 30000, 8, hyq.FMT_FP8),
    ("int4_b2_g5_w100", 2, 10, 2, 517, 100, 20000, 4, hyq.FMT_INT),
    ("int8_mha", 1, 3, 3, 300, 64, 50000, 8, hyq.FMT_INT),
    ("int4_g8_w128", 1, 16, 2, 1100, 128, 50000, 4, hyq.FMT_INT),
    ("int8_budget0", 1, 4, 1, 450, 96, 0, 8, hyq.FMT_INT),
    ("int4_all_vertical", 1, 4, 1, 200, 64, 1000000, 4, hyq.FMT_INT),
    ("fp8_window_only", 1, 4, 1, 64, 64, 50000, 8, hyq.FMT_FP8),
    ("fp4_g4", 1, 8, 2, 700, 64, 30000, 4, hyq.FMT_FP4),
    ("fp4_b2_g5_w100", 2, 10, 2, 517, 100, 20000, 4, hyq.FMT_FP4),
    ("fp4_g8_w128", 1, 16, 2, 1100, 128, 50000, 4, hyq.FMT_FP4),
]


def _inputs(name, B, Hq, Hkv, N, W, seed=0):
    return gen.generate(seed, zlib.crc32(name.encode()) % 10007 + 20000, B=B, Hq=Hq, Hkv=Hkv,
                        L=N, D=128, W=W, plant=0.03)


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_decode_small(case):
    """Freeze, then 140 appended tokens (two merges, the ring wrapping),
    with the whole cache and the attention output checked along the way."""
    name, B, Hq, Hkv, N, W, ppm, bits, fmt = case
    print(f"case {name}", flush=True)
    shape = hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=N, window=W, budget_ppm=ppm, bits_kv=bits,
                      kv_format=fmt)
    d = _inputs(name, B, Hq, Hkv, N, W)
    cache, oc = freeze_both(shape, d, N + 200)
    check_cache(cache, oc)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    check_attention(cache, oc, rng, label=name)
    for step in range(1, 141):
        append_both(cache, oc, rng)
        if step in (1, 63, 64, 65, 66, 128, 129, 140):
            check_attention(cache, oc, rng, label=name)
    assert cache.c.n_merged == 2 and cache.c.n_staged == 12
    check_cache(cache, oc)


def test_decode_bf16_output_and_deterministic():
    import torch
    shape = hyq.Shape(B=1, Hq=8, Hkv=2, L=900, window=128, budget_ppm=50000, bits_kv=4)
    d = _inputs("det", 1, 8, 2, 900, 128)
    cache, oc = freeze_both(shape, d, 1000)
    rng = np.random.default_rng(3)
    for _ in range(70):
        append_both(cache, oc, rng)
    check_attention(cache, oc, np.random.default_rng(4), out_dtype=1, label="bf16")
    q = gc.to_dev(_rows(np.random.default_rng(5), 1, 8))
    outs = []
    for _ in range(2):
        o = torch.empty((1, 8, 128), dtype=torch.float32, device="cuda")
        hyq.hyq_decode_attn(cache, q, o)
        outs.append(o.cpu().numpy())
    np.testing.assert_array_equal(outs[0], outs[1])


def test_decode_cache_full_is_an_error():
    import torch
    N, W = 300, 64
    shape = hyq.Shape(B=1, Hq=4, Hkv=1, L=N, window=W, budget_ppm=20000, bits_kv=8)
    d = _inputs("full", 1, 4, 1, N, W)
    cache, oc = freeze_both(shape, d, N + 64)       # room for one merge
    rng = np.random.default_rng(6)
    for _ in range(128):
        append_both(cache, oc, rng)
    before = cache.state
    kn = gc.to_dev(_rows(rng, 1, 1))
    with pytest.raises(hyq.HyqError) as e:
        hyq.hyq_decode_append(cache, kn, kn)
    assert e.value.code == hyq.HYQ_EINVAL and "full" in str(e.value)
    assert cache.state == before
    torch.cuda.synchronize()
    check_cache(cache, oc)
    check_attention(cache, oc, rng, label="full")


# (name, B, Hq, Hkv, N, W, budget_ppm, bits, fmt, staging)
STAGING = [
    ("int4_ws128", 1, 8, 2, 700, 128, 30000, 4, hyq.FMT_INT, 128),
    ("fp8_ws128_w200", 2, 10, 2, 517, 200, 20000, 8, hyq.FMT_FP8, 128),
    ("fp4_ws192_w200", 1, 16, 2, 1100, 200, 50000, 4, hyq.FMT_FP4, 192),
]


@pytest.mark.parametrize("case", STAGING, ids=[c[0] for c in STAGING])
def test_decode_staging_capacity(case):
    """A staging buffer of W_s = 128 or 192 tokens: a full one merges W_s/64
    blocks at once (oldest first); 2 * W_s + 5 appended tokens, the cache and
    the attention output checked around each merge."""
    name, B, Hq, Hkv, N, W, ppm, bits, fmt, ws = case
    print(f"case {name}", flush=True)
    shape = hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=N, window=W, budget_ppm=ppm, bits_kv=bits,
                      kv_format=fmt, staging=ws)
    d = _inputs(name, B, Hq, Hkv, N, W)
    cache, oc = freeze_both(shape, d, N + 3 * ws)
    assert cache.c.staging == ws
    check_cache(cache, oc)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    for step in range(1, 2 * ws + 6):
        append_both(cache, oc, rng)
        if step in (1, ws, ws + 1, ws + 2, 2 * ws + 1, 2 * ws + 5):
            check_attention(cache, oc, rng, label=name)
            if step in (ws + 1, 2 * ws + 1):
                check_cache(cache, oc)
    assert cache.c.n_merged == 2 * (ws // 64) and cache.c.n_staged == 5
    check_cache(cache, oc)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("bits,fmt,ws", [(4, hyq.FMT_INT, 128), (4, hyq.FMT_FP4, 64),
                                         (8, hyq.FMT_INT, 128)],
                         ids=["int4_ws128", "fp4_ws64", "int8_ws128"])
def test_decode_32k_k4v4_top5_w128(bits, fmt, ws):
    """The paper's decode-latency workload: batch 1, 32 query / 8 KV heads,
    d 128, 32k-token prefix, K4V4, top-5% vertical lines, window 128 (with
    the 128-token staging buffer the benchmark uses, and with the default);
    also with 8-bit codes.  On a 256-CU device all three launch one
    workgroup per CU with uneven shares of the quantized blocks, and the
    8-bit one gives each full-precision wave two tiles."""
    N, W = 32768, 128
    shape = hyq.Shape(B=1, Hq=32, Hkv=8, L=N, window=W, budget_ppm=50000, bits_kv=bits,
                      kv_format=fmt, staging=ws)
    print("generating", flush=True)
    d = gen.generate(0, 7, B=1, Hq=32, Hkv=8, L=N, D=128, W=W, plant=0.05,
                     outliers=(3, 47, 85, 122))
    print("freeze (GPU and oracle)", flush=True)
    cache, oc = freeze_both(shape, d, N + 256)
    print("comparing the cache", flush=True)
    check_cache(cache, oc)
    rng = np.random.default_rng(77)
    check_attention(cache, oc, rng, label="32k")
    for _ in range(ws + 1):                  # the last append merges the staging buffer
        append_both(cache, oc, rng)
    assert cache.c.n_merged == ws // 64
    check_attention(cache, oc, rng, label="32k")
    check_cache(cache, oc)


@pytest.mark.timeout(300)
def test_decode_batch4_reshaped_split():
    """Batch 4, 32 query / 8 KV heads, 4k prefix, int8: the default split
    (320 workgroups) is cut to one workgroup per CU on a 256-CU device, each
    wave taking 2 or 3 consecutive quantized blocks; checked through one merge."""
    name, B, Hq, Hkv, N, W = "b4_reshaped", 4, 32, 8, 4096, 128
    print(f"case {name}", flush=True)
    shape = hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=N, window=W, budget_ppm=50000, bits_kv=8)
    d = _inputs(name, B, Hq, Hkv, N, W)
    cache, oc = freeze_both(shape, d, N + 128)
    check_cache(cache, oc)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    check_attention(cache, oc, rng, label=name)
    for _ in range(65):
        append_both(cache, oc, rng)
    assert cache.c.n_merged == 1
    check_attention(cache, oc, rng, label=name)


def test_decode_attention_in_a_hip_graph():
    """Decode attention captured in a HIP graph (as a decode loop runs it):
    each replay, with eager work and synchronizations in between, equals the
    eager result bit for bit."""
    import torch
    shape = hyq.Shape(B=2, Hq=8, Hkv=2, L=800, window=64, budget_ppm=30000, bits_kv=4)
    d = _inputs("graph", 2, 8, 2, 800, 64)
    cache, oc = freeze_both(shape, d, 900)
    rng = np.random.default_rng(8)
    for _ in range(70):
        append_both(cache, oc, rng)
    q = gc.to_dev(_rows(rng, 2, 8))
    out = torch.empty((2, 8, 128), dtype=torch.float32, device="cuda")
    hyq.hyq_decode_attn(cache, q, out)
    torch.cuda.synchronize()
    ref = out.clone()
    O = orc.decode_attention(q.view(torch.int16).cpu().numpy().view(np.uint16), oc)
    mx, mean = gc.attention_error(ref.cpu().numpy(), O)
    assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        hyq.hyq_decode_attn(cache, q, out)
    for i in range(4):
        out.fill_(float("nan"))
        junk = torch.randn(1 << 20, device="cuda").sum()     # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {i}"
        del junk
