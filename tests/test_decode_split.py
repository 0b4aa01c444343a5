"""Host-side decode launch shape (`decode_split.h`): the choices for the
benchmark's decode workloads and the invariants every choice keeps.

The header is plain C++; it is compiled here with g++ beside a small driver
(`decode_split_check.cpp`), so these run without a GPU.
"""
import math
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2608_27875_amd", "csrc")


@pytest.fixture(scope="module")
def split_tool(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("split") / "split_check")
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", CSRC,
                    os.path.join(HERE, "decode_split_check.cpp"), "-o", exe], check=True)

    def run(cases):
        inp = "".join(f"{nbq} {nft} {heads} {n_cu} {bits}\n" for nbq, nft, heads, n_cu, bits in cases)
        out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout
        return [tuple(int(x) for x in line.split()) for line in out.splitlines()]
    return run


def _default(nbq, nft, bits):
    u = 4 if bits == 4 else 2
    return math.ceil(nbq / (4 * u)), math.ceil(nft / 4)


def _busiest_bytes(nbq, nft, heads, n_cu, bits, s_q, s_f):
    """Bytes of the busiest SIMD: workgroups on the busiest CU x bytes of the
    busiest wave (4 waves per workgroup)."""
    blk, tile = 2 * 64 * 128 * bits // 8, 2 * 64 * 128 * 2
    per_cu = math.ceil((s_q + s_f) * heads / n_cu)
    wave = max(math.ceil(nbq / (4 * s_q)) * blk if s_q else 0,
               math.ceil(nft / (4 * s_f)) * tile if s_f else 0)
    return per_cu * wave


# 32k prefix, top-5%, W = 128, W_s = 128: 485 quantized blocks and 30
# full-precision tiles per KV head, 8 KV heads per sequence
BENCH = (485, 30)


@pytest.mark.parametrize("heads,bits,expect", [
    (8, 4, (24, 8)),      # batch 1: one workgroup per CU, 5-6 int4 blocks per wave
    (8, 8, (28, 4)),      # batch 1, 8-bit: two full-precision tiles per wave
    (16, 4, (12, 4)),     # batch 2
    (32, 4, (31, 8)),     # batch 4: the default (about five workgroups per CU)
    (128, 4, (31, 8)),    # batch 16: the default
])
def test_benchmark_shapes(split_tool, heads, bits, expect):
    assert split_tool([(*BENCH, heads, 256, bits)]) == [expect]


def test_candidates_are_bounded_by_the_default_split(split_tool):
    """Every candidate shape is capped by the default split, not by a
    candidate found earlier in the search (two cases where the two differ)."""
    assert split_tool([(485, 10, 16, 256, 4), (1000, 5, 24, 256, 4)]) == [(14, 2), (51, 2)]


def test_default_when_it_fits_or_nothing_is_quantized(split_tool):
    assert split_tool([(*BENCH, 8, 1024, 4)]) == [_default(*BENCH, 4)]   # 312 <= 1024 CUs
    assert split_tool([(0, 30, 8, 256, 4)]) == [(0, 8)]
    assert split_tool([(2, 30, 8, 256, 4)]) == [_default(2, 30, 4)]


def test_invariants_over_a_grid(split_tool):
    cases = [(nbq, nft, heads, n_cu, bits)
             for nbq in (1, 7, 64, 485, 2000)
             for nft in (1, 5, 30, 200)
             for heads in (1, 3, 8, 16, 40, 128)
             for n_cu in (80, 256, 304)
             for bits in (4, 8)]
    got = split_tool(cases)
    assert len(got) == len(cases)
    for (nbq, nft, heads, n_cu, bits), (s_q, s_f) in zip(cases, got):
        dq, df = _default(nbq, nft, bits)
        # never more splits than the default (the workspace is sized for it)
        assert 1 <= s_q <= dq and 1 <= s_f <= df, (nbq, nft, heads, n_cu, bits, s_q, s_f)
        # a reshaped launch has no busier SIMD than the default one
        assert (_busiest_bytes(nbq, nft, heads, n_cu, bits, s_q, s_f)
                <= _busiest_bytes(nbq, nft, heads, n_cu, bits, dq, df))
        # when the default already fits the CUs, it is kept
        if (dq + df) * heads <= n_cu:
            assert (s_q, s_f) == (dq, df)
