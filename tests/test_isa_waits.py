"""Every MFMA result in the library's gfx950 code waits as long on every
control-flow path as on a straight one (see isa_waits.py for why this is
checked)."""
import os
import shutil
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2608_27875_amd import build as hyq_build
from tests.isa_waits import device_asm, short_paths

HIP_SOURCES = [s for s in hyq_build.SOURCES if s.endswith(".hip")]

# A reduced form of a loop whose last MFMA was followed by a conditional block
# before its result was read: the path that skips the block was left short.
_SHORT = """
_k:
  v_mfma_f32_32x32x16_bf16 a[0:15], v[2:5], v[6:9], a[0:15]
  s_cbranch_vccnz .LBB0_2
  v_subrev_u32_e32 v2, 31, v58
  v_cmp_le_i32_e32 vcc, v2, v52
  v_cmp_gt_i32_e64 s[0:1], s7, v2
  s_and_b64 s[0:1], vcc, s[0:1]
  s_orn2_b64 s[0:1], s[0:1], exec
.LBB0_2:
  s_nop 5
  v_accvgpr_read_b32 v17, a15
  s_endpgm
_j:
  v_mfma_f32_32x32x16_bf16 a[0:15], v[2:5], v[6:9], a[0:15]
  s_nop 10
  v_accvgpr_read_b32 v17, a15
  s_endpgm
"""


def test_checker_flags_short_path():
    bad, need = short_paths(_SHORT)
    assert need[("v_mfma_f32_32x32x16_bf16", "other")] == 11
    assert [(b[0], b[3]) for b in bad] == [("_k", 7)]


def test_checker_accepts_straight_line():
    bad, _ = short_paths("_j:" + _SHORT.split("_j:")[1])
    assert bad == []


@pytest.mark.skipif(shutil.which(hyq_build.HIPCC) is None and not os.path.exists(hyq_build.HIPCC),
                    reason="hipcc not available")
def test_library_mfma_waits():
    srcs = [os.path.join(hyq_build.CSRC, s) for s in HIP_SOURCES]
    with ThreadPoolExecutor(max_workers=4) as ex:
        asms = list(ex.map(lambda p: device_asm(p, hyq_build.HIPCC, hyq_build.FLAGS), srcs))
    problems = []
    for src, asm in zip(HIP_SOURCES, asms):
        bad, _ = short_paths(asm)
        problems += [f"{src}: {fn}: {t} ({kind} reader after {mn} < {n} wait states)"
                     for fn, t, kind, mn, n in bad]
    assert not problems, "\n".join(problems[:20])
