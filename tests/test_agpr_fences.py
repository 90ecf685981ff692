"""The 4-wave GEMM keeps its accumulators in AGPRs through inline-asm MFMAs,
which the compiler's hazard recognizer does not see: its assembly must give
every MFMA's result registers their wait states on every path, including
the register copies and spill code the compiler places at loop edges.
Compiles k_gemm.hip to assembly (CPU only)."""

import os
import shutil

import pytest

from paper_2608_26140_amd import check_agpr_fences as chk
from paper_2608_26140_amd.build import HIPCC


def _have_hipcc():
    return os.path.exists(HIPCC) or shutil.which(HIPCC) is not None


@pytest.mark.skipif(not _have_hipcc(), reason="hipcc not found")
def test_gemm_agpr_wait_states(capsys):
    rc = chk.main([])
    out = capsys.readouterr().out
    assert rc == 0, out
    assert "checked 5 kernels" in out


def test_checker_flags_unfenced_reads():
    # an accumulator read 3 instructions after an MFMA, reached over a branch
    asm = """
	v_mfma_f32_16x16x32_bf16 a[0:3], v[0:3], v[4:7], a[0:3]
	s_cbranch_scc1 .LBB0_2
	s_nop 7
	s_nop 7
	s_nop 7
.LBB0_2:
	v_accvgpr_read_b32 v8, a0
	s_endpgm
""".splitlines()
    bad = chk.unfenced(asm)
    assert len(bad) == 1 and "v_accvgpr_read" in bad[0][1]
    # fenced on both paths
    ok = asm[:2] + ["\ts_nop 7", "\ts_nop 7", "\ts_nop 7"] + asm[2:]
    assert chk.unfenced(ok) == []


def test_checker_flags_write_before_mfma():
    asm = """
	v_accvgpr_write_b32 a0, 0
	v_mfma_f32_16x16x32_bf16 a[0:3], v[0:3], v[4:7], a[0:3]
	s_nop 7
	s_nop 7
	s_nop 7
	s_endpgm
""".splitlines()
    bad = chk.unfenced(asm)
    assert len(bad) == 1 and "v_mfma" in bad[0][1]
