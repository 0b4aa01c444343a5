"""The decode cache's size against the paper's memory-overhead table (its
appendix on memory overhead: vertical-line tokens, local window and staging
buffer of a K4V4 cache, W = 128, 5% vertical lines, 8k and 32k prefixes).

Strict K4V4 keeps D/2 bytes of K and D/2 of V per token; a token kept in
bf16 costs 4D bytes, 3D more.  The table's components follow from that, and
the cache that hyq_dcache_init sizes (host arithmetic only) reproduces them
once its own choices are accounted for: vertical-line and ring rows padded to
whole 64-row tiles, the staging capacity (64 tokens by default, 128 as in the
table), and one float32 scale per 64-token block of K and of V."""
import os

import pytest

import paper_2608_27875_amd as hyq

HERE = os.path.dirname(os.path.abspath(__file__))
D = 128


def _table():
    rows = {}
    with open(os.path.join(HERE, "golden", "memory_overhead.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, a, b = line.split()
                rows[name] = {8192: float(a), 32768: float(b)}
    return rows


@pytest.mark.parametrize("N", [8192, 32768])
def test_components_follow_the_bf16_vs_k4v4_cost(N):
    t = _table()
    W, r = 128, 0.05
    extra = 3 * D                              # bf16 K+V (4D) minus K4V4 (D) per token
    assert 100 * r * extra / D == pytest.approx(t["vl_tokens"][N], abs=0.05)
    assert 100 * W * extra / (N * D) == pytest.approx(t["local_window"][N], abs=0.05)
    assert 100 * 128 * extra / (N * D) == pytest.approx(t["staging_buffer"][N], abs=0.05)
    total = t["vl_tokens"][N] + t["local_window"][N] + t["staging_buffer"][N]
    assert total == pytest.approx(t["total"][N], abs=0.15)


@pytest.mark.parametrize("N", [8192, 32768])
@pytest.mark.parametrize("Ws", [hyq.DECODE_WS, 128])
def test_cache_sizes_reproduce_the_table(N, Ws):
    """Overhead of the cache hyq_dcache_init sizes for a Freeze of N tokens
    (no appended token yet), split into the table's components plus this
    layout's padding and scales; with the table's 128-token staging buffer
    and with the default 64."""
    t = _table()
    W, ppm = 128, 50000
    shape = hyq.Shape(B=1, Hq=32, Hkv=8, L=N, window=W, budget_ppm=ppm, bits_kv=4, staging=Ws)
    c, z = hyq.hyq_dcache_init(shape, N)
    Hkv = 8
    strict = Hkv * N * D                       # K4V4 bytes of N tokens
    k = c.n_vl
    nq = c.n_frozen
    codes = z["k_codes_bytes"] + z["v_codes_bytes"]
    assert codes == Hkv * c.cap_blocks * 64 * D           # D/2 + D/2 bytes per slot
    scales = z["k_scale_bytes"] + z["v_scale_bytes"]
    fp = z["fp_k_bytes"] + z["fp_v_bytes"]
    assert fp == Hkv * (c.vl_rows + c.ring_rows) * 4 * D  # bf16 K and V rows
    # the table's components, from this cache's own token counts
    vl = Hkv * k * 3 * D
    win = Hkv * W * 3 * D
    staged = Hkv * Ws * 4 * D                  # empty staging rows (tokens yet to come)
    pad_vl = Hkv * (c.vl_rows - k) * 4 * D
    pad_ring = Hkv * (c.ring_rows - W - Ws) * 4 * D
    pad_blk = Hkv * (c.cap_blocks * 64 - nq) * D
    assert nq + k + W == N
    total = codes + scales + fp
    assert total - strict == vl + win + staged + pad_vl + pad_ring + pad_blk + scales
    pct = lambda x: 100.0 * x / strict
    # vertical lines: k = ceil(5% of the N - W prefix tokens), so slightly under 15%
    assert pct(vl) == pytest.approx(t["vl_tokens"][N], abs=0.3)
    assert pct(win) == pytest.approx(t["local_window"][N], abs=0.05)
    # the table prices staged tokens at 3D (bf16 instead of K4V4); rows for
    # tokens not yet appended cost their whole 4D
    assert pct(staged) == pytest.approx(t["staging_buffer"][N] * Ws / 128 * 4 / 3, abs=0.05)
    # this layout's own additions stay small
    assert pct(pad_vl + pad_ring + pad_blk + scales) < 2.5
