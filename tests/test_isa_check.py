"""The static check on the image GEMM's untracked filter loads
(paper_1903_06934_amd/isa_check.py): it accepts the built kernels and
rejects each kind of violation planted into a small loop."""
import os

import pytest

from paper_1903_06934_amd import build, isa_check

# Three pipeline stages: stage 1 consumes v[2:5] and loads v[10:13], stage 2
# consumes v[6:9] and loads v[2:5], stage 3 consumes v[10:13] and loads
# v[6:9]; v3 is used as a temporary between its last use and its next load.
LOOP = """_ZN6miconv15img_gemm_kernelILi64EEvNS_11ImgGemmArgsE:
\ts_mov_b32 s0, 0
.LBB0_1:                               ; =>This Inner Loop Header: Depth=1
\ts_waitcnt vmcnt(5)
\ts_barrier
\tv_mfma_f32_16x16x4_f32 a[0:3], v2, v30, a[0:3]
\tv_add_u32_e32 v3, 4, v21
\tbuffer_load_dwordx4 v[10:13], v3, s[0:3], 0 offen
\ts_waitcnt vmcnt(5)
\ts_barrier
\tv_mfma_f32_16x16x4_f32 a[0:3], v6, v30, a[0:3]
\tbuffer_load_dwordx4 v[2:5], v21, s[0:3], 0 offen
\ts_waitcnt vmcnt(5)
\ts_barrier
\tv_mfma_f32_16x16x4_f32 a[0:3], v10, v30, a[0:3]
\tbuffer_load_dwordx4 v[6:9], v22, s[0:3], 0 offen
\ts_cbranch_scc1 .LBB0_1
.Lfunc_end0:
"""


def test_clean_loop_passes():
    assert isa_check.check_assembly(LOOP) == []


@pytest.mark.parametrize("old,new,what", [
    # a use one stage after the load: still in flight
    ("\tv_mfma_f32_16x16x4_f32 a[0:3], v6, v30, a[0:3]",
     "\tv_mfma_f32_16x16x4_f32 a[0:3], v10, v30, a[0:3]", "in flight"),
    # a copy of a loaded register before its use
    ("\tv_mfma_f32_16x16x4_f32 a[0:3], v2, v30, a[0:3]",
     "\tv_mov_b32_e32 v40, v2\n\tv_mfma_f32_16x16x4_f32 a[0:3], v2, v30, a[0:3]", "only v_mfma"),
    # a temporary written into a register before its last use
    ("\tv_mfma_f32_16x16x4_f32 a[0:3], v2, v30, a[0:3]",
     "\tv_add_u32_e32 v2, 4, v21\n\tv_mfma_f32_16x16x4_f32 a[0:3], v2, v30, a[0:3]",
     "before its last use"),
])
def test_planted_violations_fail(old, new, what):
    assert old in LOOP
    errors = isa_check.check_assembly(LOOP.replace(old, new, 1))
    assert any(what in e for e in errors), errors


def test_built_kernels_pass():
    src = os.path.join(build.CSRC, "conv_kernels.hip")
    text = isa_check.compile_assembly(build.HIPCC, build.FLAGS, src)
    assert isa_check.check_assembly(text) == []
