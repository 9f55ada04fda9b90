"""The two-group attention kernel issues its MFMAs as inline assembly, so the
compiler does not keep the matrix cores' dependency distances around them;
the kernel's source does (explicit wait states, and empty register
constraints that pin where VALU results are produced and how long MFMA
operands stay live).  These tests compile ``attention.hip`` to gfx950
assembly and check every instance of that kernel for the three hazard
patterns of ``tests/mfma_hazards.py``; the checker itself is first shown to
flag hand-made cases of each pattern and to pass their corrected forms."""
import os
import shutil
import subprocess

import pytest

from tests import mfma_hazards as mh

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2607_06631_amd", "csrc", "attention.hip")
G2_KERNELS = [
    "_ZN3dif20flash_attn_g2_kernelILb1EEEvNS_10AttnParamsIDF16bEE",
    "_ZN3dif20flash_attn_g2_kernelILb0EEEvNS_10AttnParamsIDF16bEE",
]

MFMA_NEGM = "v_mfma_f32_32x32x16_bf16 v[50:65], v[82:85], a[156:159], v[2:17]"


def kinds(lines):
    return sorted({h.kind for h in mh.scan_lines(lines)})


def test_checker_flags_valu_write_before_mfma_operand():
    bad = ["v_mov_b32_e32 v17, v2", MFMA_NEGM]
    assert kinds(bad) == ["A"]
    assert kinds(["v_mov_b32_e32 v17, v2", "s_nop 1", MFMA_NEGM]) == []
    # an A/B operand counts as well
    assert kinds(["v_cvt_pk_bf16_f32 v84, v1, v2", MFMA_NEGM]) == ["A"]


def test_checker_flags_early_read_of_mfma_result():
    seq = [MFMA_NEGM, "v_add_f32_e32 v1, v1, v1", "v_exp_f32_e32 v66, v50"]
    assert kinds(seq) == ["B"]
    assert kinds([MFMA_NEGM, "s_nop 15", "v_exp_f32_e32 v66, v50"]) == []
    # two MFMAs in between cover it (each waits for the previous one's passes)
    other = "v_mfma_f32_32x32x16_bf16 a[0:15], v[90:93], v[94:97], a[0:15]"
    assert kinds([MFMA_NEGM, other, other, "v_exp_f32_e32 v66, v50"]) == []
    # an LDS write of the result is a read too
    assert kinds([MFMA_NEGM, "ds_write_b64 v3, v[50:51]"]) == ["B"]


def test_checker_flags_reuse_of_accumulator_input():
    seq = [MFMA_NEGM, "v_exp_f32_e32 v14, v40"]
    assert kinds(seq) == ["C"]
    assert kinds([MFMA_NEGM, "s_nop 7", "v_exp_f32_e32 v14, v40"]) == []


def test_checker_follows_branches_and_loops():
    # the write sits before a branch, the MFMA at its target
    seq = ["s_cbranch_scc0 .LBB0_3", "v_mov_b32_e32 v2, 0", "s_branch .LBB0_2",
           ".LBB0_3:", "v_mov_b32_e32 v3, 0", "s_nop 4", ".LBB0_2:", MFMA_NEGM, "s_endpgm"]
    assert kinds(seq) == ["A"]
    # a loop: the MFMA at the bottom, its result read at the top
    loop = [".LBB0_1:", "v_exp_f32_e32 v66, v50", "v_add_f32_e32 v1, v1, v1", MFMA_NEGM,
            "s_cbranch_scc1 .LBB0_1", "s_endpgm"]
    assert kinds(loop) == ["B"]


@pytest.fixture(scope="module")
def attention_asm(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    from paper_2607_06631_amd import build
    out = tmp_path_factory.mktemp("asm") / "attention.s"
    flags = [f for f in build.FLAGS if f != "-fPIC"]
    cmd = [hipcc, *flags, "--cuda-device-only", "-S", SRC, "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


@pytest.mark.parametrize("kernel", G2_KERNELS)
def test_two_group_kernel_keeps_mfma_distances(attention_asm, kernel):
    hz = mh.scan(attention_asm, kernel)
    assert not hz, "\n".join(f"{h.kind} ({h.wait_states} wait states): {h.first} -> {h.second}" for h in hz)
