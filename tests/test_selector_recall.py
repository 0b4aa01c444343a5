"""How well the two selectors of Section 4.1 find vertical lines that the
attention itself makes (gen.shared_direction: every query of a KV group
carries a shared direction, and the planted keys lie along it, so each planted
key gets the same logit boost from every query).  The oracle's Algorithm 1
(summed tail queries, eq. vl_topk) and its exact column mass (eq. vl_score)
must both recover most planted lines, and fewer when the lines are weak.
These are properties of the method on such inputs, not parity pins."""
import numpy as np
import pytest

from oracle import hyq_oracle as orc
from paper_2608_27875_amd import gen

B, HQ, HKV, L, W, PPM = 1, 8, 2, 4096, 128, 20000


def recall(idx, planted, P, k):
    out = []
    for bj, pos in enumerate(planted):
        pp = set(p for p in pos.tolist() if p < P)
        out.append(len(pp & set(idx.reshape(-1, k)[bj].tolist())) / min(len(pp), k))
    return float(np.mean(out))


def both(alpha, beta):
    d = gen.shared_direction(0, B=B, Hq=HQ, Hkv=HKV, L=L, D=128, W=W, plant=0.01,
                             alpha=alpha, beta=beta)
    sz = orc.sizes(L, W, PPM)
    i1, _ = orc.select_vertical(d["Q"], d["K"], HKV, W, PPM)
    i2, _ = orc.select_vertical_colmass(d["Q"], d["K"], HKV, W, PPM)
    return (recall(i1, d["planted"], sz["P"], sz["k"]),
            recall(i2, d["planted"], sz["P"], sz["k"]))


def test_shared_direction_inputs_are_deterministic_and_planted():
    a = gen.shared_direction(3, B=1, Hq=4, Hkv=1, L=256, D=128, W=32, plant=0.02)
    b = gen.shared_direction(3, B=1, Hq=4, Hkv=1, L=256, D=128, W=32, plant=0.02)
    for key in ("Q", "K", "V"):
        np.testing.assert_array_equal(a[key], b[key])
    pos = a["planted"][0]
    assert pos[0] == 0 and len(pos) == 1 + round(0.02 * 256) and np.all(np.diff(pos) > 0)


def test_both_selectors_find_strong_lines():
    r_proxy, r_mass = both(7.0, 4.0)
    print(f"strong lines: tail proxy {r_proxy:.3f}, column mass {r_mass:.3f}")
    assert r_proxy >= 0.8 and r_mass >= 0.7


def test_weaker_lines_are_found_less_often():
    strong, weak = both(7.0, 4.0), both(4.0, 2.0)
    print(f"tail proxy {strong[0]:.3f} -> {weak[0]:.3f}, column mass {strong[1]:.3f} -> {weak[1]:.3f}")
    assert weak[0] < strong[0] and weak[1] < strong[1]
