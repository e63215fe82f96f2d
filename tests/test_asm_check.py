"""The build-time check of kernels whose LDS reads are inline assembly
(paper_2403_11366_amd/asm_check.py): planted hazards in small assembly
listings are found, the safe pattern passes, and the built library's saved
gfx950 assembly passes (when it has been built here)."""
import glob
import os

import pytest

from paper_2403_11366_amd import asm_check

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _fn(body: str) -> str:
    return "_Z4testv:\n" + body + "\n.Lfunc_end0:\n"


SAFE = """
	;;#ASMSTART
	ds_read_b128 v[10:13], v1 offset:0
	;;#ASMEND
	;;#ASMSTART
	ds_read_b128 v[14:17], v1 offset:4096
	;;#ASMEND
	;;#ASMSTART
	s_waitcnt lgkmcnt(1)
	;;#ASMEND
	v_mfma_f32_32x32x16_bf16 v[20:35], v[10:13], v[40:43], v[20:35]
	;;#ASMSTART
	s_waitcnt lgkmcnt(0)
	;;#ASMEND
	v_mfma_f32_32x32x16_bf16 v[20:35], v[14:17], v[40:43], v[20:35]
	s_barrier
"""


def test_safe_pattern_passes():
    assert asm_check.check_assembly(_fn(SAFE)) == []


def test_use_before_the_covering_wait_is_found():
    # the second read's registers used after a wait that retires only the first
    bad = SAFE.replace("v[10:13], v[40:43]", "v[14:17], v[40:43]", 1)
    errs = asm_check.check_assembly(_fn(bad))
    assert errs and "before its LDS read completed" in errs[0]


def test_copy_of_a_pending_destination_is_found():
    bad = SAFE.replace("\t;;#ASMSTART\n\ts_waitcnt lgkmcnt(1)", "\tv_mov_b32_e32 v50, v11\n\t;;#ASMSTART\n\ts_waitcnt lgkmcnt(1)", 1)
    assert asm_check.check_assembly(_fn(bad))


def test_scratch_and_calls_are_found():
    assert asm_check.check_assembly(_fn(SAFE + "\tscratch_store_dword off, v3, off offset:4\n"))
    assert asm_check.check_assembly(_fn(SAFE + "\ts_swappc_b64 s[30:31], s[16:17]\n"))


def test_pending_read_at_a_branch_is_found():
    bad = SAFE.replace("\t;;#ASMSTART\n\ts_waitcnt lgkmcnt(1)", "\ts_cbranch_scc1 .LBB0_2\n\t;;#ASMSTART\n\ts_waitcnt lgkmcnt(1)", 1)
    assert any("branch" in e for e in asm_check.check_assembly(_fn(bad)))


def test_functions_without_asm_reads_are_ignored():
    body = "\tds_read_b128 v[10:13], v1\n\tv_mov_b32_e32 v50, v11\n\tscratch_store_dword off, v3, off\n"
    assert asm_check.check_assembly(_fn(body)) == []


def test_built_library_assembly_passes():
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2403_11366_amd", "_build", "*-hip-amdgcn-amd-amdhsa-gfx950.s")))
    if not files:
        pytest.skip("library not built here")
    assert asm_check.check_files(files) == []
    assert asm_check.count_checked(files) >= 1


# One asm block that forms its addresses and then issues the reads (the form of
# the 256x256 forward tile's reads): the reads inside the block are tracked.
XOR_BLOCK = """
	;;#ASMSTART
	v_xor_b32 v2, 32, v1
	v_xor_b32 v3, 32, v4
	ds_read_b128 v[10:13], v2
	ds_read_b128 v[14:17], v2 offset:4096
	ds_read_b128 v[18:21], v3
	;;#ASMEND
	;;#ASMSTART
	s_waitcnt lgkmcnt(0)
	;;#ASMEND
	v_mfma_f32_32x32x16_bf16 v[20:35], v[10:13], v[18:21], v[20:35]
"""


def test_reads_after_address_arithmetic_in_one_block():
    assert asm_check.check_assembly(_fn(XOR_BLOCK)) == []
    assert asm_check.count_checked_text(_fn(XOR_BLOCK)) == 1
    bad = XOR_BLOCK.replace("\t;;#ASMSTART\n\ts_waitcnt lgkmcnt(0)", "\tv_mov_b32_e32 v50, v15\n\t;;#ASMSTART\n\ts_waitcnt lgkmcnt(0)", 1)
    errs = asm_check.check_assembly(_fn(bad))
    assert errs and "before its LDS read completed" in errs[0]
