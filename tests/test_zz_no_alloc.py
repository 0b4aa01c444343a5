"""The allocation-free decode attention call (hyq_decode_attn_noalloc)
against hyq_decode_attn with a workspace, through the C ABI: the same
kernels, so the outputs must agree bit for bit; both also against the
oracle's decode attention (max-abs 2e-3, mean-abs 2e-4).  Two calls in a
row, the second on a smaller cache, so that the shared scratch's contents
from the first call cannot leak into the second.  Also the size limit."""
import numpy as np
import pytest

import gpu_common as gc
import paper_2608_27875_amd as hyq
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen

pytestmark = pytest.mark.gpu


def _cache(seed, B, Hq, Hkv, N, W, ppm, bits, n_append, fmt=hyq.FMT_INT):
    import torch
    d = gen.generate(seed, 9100 + seed, B=B, Hq=Hq, Hkv=Hkv, L=N, D=128, W=W, plant=0.05)
    shape = hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=N, window=W, budget_ppm=ppm, bits_kv=bits,
                      kv_format=fmt)
    dev = torch.device("cuda:0")
    cache = hyq.DecodeCache(shape, N + n_append + 64, dev)
    hyq.hyq_freeze(shape, gc.to_dev(d["Q"]), gc.to_dev(d["K"]), gc.to_dev(d["V"]), cache)
    oc = orc.freeze(d["Q"], d["K"], d["V"], Hkv, W, ppm, bits, fmt=gc.fmt_name(shape))
    rng = np.random.default_rng(seed)
    for _ in range(n_append):
        kv = [gen.f32_to_bf16_bits(rng.standard_normal((B, Hkv, 128)).astype(np.float32))
              for _ in range(2)]
        hyq.hyq_decode_append(cache, gc.to_dev(kv[0]), gc.to_dev(kv[1]))
        orc.decode_append(oc, kv[0], kv[1])
    q = gen.f32_to_bf16_bits(rng.standard_normal((B, Hq, 128)).astype(np.float32))
    return cache, oc, q


def _both(cache, q):
    import torch
    c = cache.c
    qd = gc.to_dev(q)
    o_ws = torch.full((c.B, c.Hq, 128), float("nan"), dtype=torch.float32, device=qd.device)
    o_na = torch.full_like(o_ws, float("nan"))
    hyq.hyq_decode_attn_noalloc(cache, qd, o_na)
    hyq.hyq_decode_attn(cache, qd, o_ws)
    torch.cuda.synchronize()
    return o_ws.cpu().numpy(), o_na.cpu().numpy()


def test_noalloc_matches_workspace_call_twice():
    # first call: batch 2, int4, a merge behind it; second: a smaller cache
    for case in ((1, 2, 8, 2, 900, 128, 50000, 4, 70), (2, 1, 4, 1, 300, 64, 30000, 8, 5)):
        seed, B, Hq, Hkv, N, W, ppm, bits, n_app = case
        print(f"noalloc case B={B} Hq={Hq} Hkv={Hkv} N={N} bits={bits} appended={n_app}", flush=True)
        cache, oc, q = _cache(seed, B, Hq, Hkv, N, W, ppm, bits, n_app)
        o_ws, o_na = _both(cache, q)
        np.testing.assert_array_equal(o_na.view(np.uint32), o_ws.view(np.uint32))
        ref = orc.decode_attention(q, oc)
        mx, mean = gc.attention_error(o_na, ref)
        print(f"  max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
        assert mx <= gc.TOL_MAX and mean <= gc.TOL_MEAN


def test_noalloc_rejects_launch_beyond_scratch():
    """A cache whose partials exceed the scratch is refused before anything
    is enqueued (the workspace call still works)."""
    import torch
    shape = hyq.Shape(B=64, Hq=32, Hkv=8, L=32768, window=128, budget_ppm=50000, bits_kv=4)
    c, _ = hyq.hyq_dcache_init(shape, 32768 + 64)
    cache = hyq.DecodeCache.__new__(hyq.DecodeCache)
    cache.c, cache.device = c, torch.device("cuda:0")
    for n in ("k_codes", "v_codes", "k_scale", "v_scale", "q_pos", "fp_k", "fp_v", "vl_pos"):
        setattr(c, n, 256)   # never dereferenced: the call fails before any launch
    q = torch.zeros((64, 32, 128), dtype=torch.bfloat16, device="cuda:0")
    o = torch.empty((64, 32, 128), dtype=torch.float32, device="cuda:0")
    with pytest.raises(hyq.HyqError) as e:
        hyq.hyq_decode_attn_noalloc(cache, q, o)
    assert e.value.code == hyq.HYQ_EUNSUPPORTED
