"""The post-build device-code check (paper_2607_21271_amd/isa_check.py).

Two miscompile shapes seen with this toolchain in the fp16 activation unpack
must be caught; correct code must pass; and the device assembly of the
current build, when present, must be clean.
"""
import os

import pytest

from paper_2607_21271_amd import build as B
from paper_2607_21271_amd import isa_check

KERNEL = "_ZN3eqk15eql_gemm_kernelILi3ELb1ELb0ELi2ELi2ELi0ELb0EEEvPKvS2_S2_Pvliiiiii:"


def _scan(body):
    return isa_check.scan_lines([KERNEL] + body.strip("\n").split("\n"))


def test_flags_unpack_writing_its_input():
    # early-clobber output given the input's register (as emitted by the compiler)
    probs = _scan("""
\t;;#ASMSTART
\tv_cvt_f32_f16_e32 v3, v3
\tv_cvt_f32_f16_sdwa v5, v3 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1
\t;;#ASMEND
""")
    assert [p[1] for p in probs] == ["clobbered_unpack", "converted_source"]


def test_flags_convert_of_overwritten_word():
    # a raw word overwritten by a conversion before its other half is read
    probs = _scan("""
\tv_cvt_f32_f16_sdwa v3, v2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1
\tv_cvt_f32_f16_e32 v5, v2
\tv_cvt_f32_f16_e32 v4, v3
""")
    assert [p[1] for p in probs] == ["converted_source"]


def test_passes_correct_unpack():
    probs = _scan("""
\tbuffer_load_dwordx2 v[2:3], v76, s[20:23], s58 offen
\ts_waitcnt vmcnt(0)
\t;;#ASMSTART
\tv_cvt_f32_f16_e32 v7, v2
\tv_cvt_f32_f16_sdwa v2, v2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1
\t;;#ASMEND
\t;;#ASMSTART
\tv_cvt_f32_f16_e32 v8, v3
\tv_cvt_f32_f16_sdwa v3, v3 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1
\t;;#ASMEND
\tv_add_f32_e32 v9, v7, v2
""")
    assert probs == []


def test_block_boundary_resets_state():
    # a word reloaded on another path: the scan is per basic block
    probs = _scan("""
\tv_add_f32_e32 v4, v1, v2
.LBB7_3:
\tv_cvt_f32_f16_e32 v5, v4
""")
    assert probs == []


def test_current_build_is_clean():
    files = isa_check.device_asm_files(B.BUILD_DIR)
    if not files:
        pytest.skip("no kept device assembly (library not built in this tree)")
    assert isa_check.check_build(B.BUILD_DIR) == files
    assert any("inst_f16" in f for f in files)


def test_flags_partial_overlap_of_wide_mfma_result():
    probs = _scan("""
\tv_mfma_f32_32x32x16_f16 v[4:19], v[30:33], v[34:37], v[0:15]
""")
    assert [p[1] for p in probs] == ["mfma_dst_overlap"]


def test_passes_in_place_and_four_register_mfma():
    probs = _scan("""
\tv_mfma_f32_32x32x16_f16 v[0:15], v[30:33], v[34:37], v[0:15]
\tv_mfma_f32_16x16x32_f16 v[52:55], v[158:161], v[208:211], v[54:57]
\tv_mfma_f32_16x16x32_f16 v[0:3], v[10:13], v[14:17], 0
""")
    assert probs == []
