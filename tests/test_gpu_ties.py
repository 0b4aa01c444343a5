"""GPU selection with exact score ties at the k-th largest value: the
lowest-position-wins rule (and -0 == +0) of Algorithm 1's top-k, checked
bit for bit against the oracle (indices and scores) on integer-valued inputs
whose tied threshold keys are spread over the whole prefix."""
import numpy as np
import pytest

import gpu_common as gc
from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen

pytestmark = pytest.mark.gpu

# (name, B, Hq, Hkv, L, W, budget_ppm): B*Hkv >= 8 and the 32k shape
SHAPES = [
    ("b2_h4_4k", 2, 8, 4, 4096, 64, 20000),
    ("ragged_b1_h8", 1, 16, 8, 3001, 77, 30000),
    ("gqa32q8kv_32k", 1, 32, 8, 32768, 256, 10000),
    ("prefix_over_32k", 1, 8, 2, 70000, 100, 20000),   # the top-k reads its scores in 3 parts
]


def _select(shape, d):
    import torch
    Q, K = gc.to_dev(d["Q"]), gc.to_dev(d["K"])
    bufs = gc.hyq.alloc_buffers(shape, Q.device)
    z = bufs["sizes"]
    scores = torch.empty(z["scores_bytes"] // 4, dtype=torch.float32, device=Q.device)
    gc.hyq.hyq_select_vertical(shape, Q, K, bufs["idx"], scores, bufs["ws"])
    torch.cuda.synchronize()
    return bufs["idx"].cpu().numpy(), scores.cpu().numpy()


@pytest.mark.timeout(300)
@pytest.mark.parametrize("kind", gen.TIE_KINDS)
@pytest.mark.parametrize("case", SHAPES, ids=[c[0] for c in SHAPES])
def test_topk_ties_bit_exact(case, kind):
    name, B, Hq, Hkv, L, W, ppm = case
    print(f"ties {name} {kind}", flush=True)
    k = orc.sizes(L, W, ppm)["k"]
    d = gen.tie_inputs(3, B, Hq, Hkv, L, W, k, kind)
    shape = gc.hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=L, window=W, budget_ppm=ppm, bits_kv=8)
    gi, gs = _select(shape, d)
    idx, S = orc.select_vertical(d["Q"], d["K"], Hkv, W, ppm)
    np.testing.assert_array_equal(gs.reshape(S.shape).view(np.uint32), S.view(np.uint32))
    np.testing.assert_array_equal(gi.reshape(idx.shape), idx)
    # the case really splits ties at the threshold
    s0 = S[0, 0] + np.float32(0.0)
    T = np.sort(s0)[::-1][k - 1]
    assert (s0 == T).sum() > k - (s0 > T).sum()
