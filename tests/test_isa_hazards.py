"""Static check of the gfx950 code object: the inline sequences of the decode
kernels that write SCC (the scalar shift-add of the stream position, the exec
narrowing of the renormalisation) declare it, so no instruction after them may
read SCC before something writes SCC again.  A violation lets a branch or
select take the inline sequence's SCC for a comparison result (one such case
turned the step loop of one-step chunks into a 2^32-iteration loop)."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2601_22787_amd import _build

SCC_READ = re.compile(r"^(s_cbranch_scc[01]|s_cselect_|s_addc_u32|s_subb_u32|s_cmov_|s_cmovk_)")
# scalar ALU instructions that write SCC (comparisons and arithmetic/logic)
SCC_WRITE = re.compile(
    r"^(s_cmp|s_bitcmp|s_add_|s_addk_|s_sub_|s_and_|s_or_|s_xor_|s_andn[12]_|s_orn[12]_|"
    r"s_nand_|s_nor_|s_xnor_|s_lshl_|s_lshr_|s_ashr_|s_bcnt[01]_|s_min_|s_max_|s_bfe_|"
    r"s_not_|s_abs_|s_cselect_|s_addc_|s_subb_|s_bitset|s_lshl[1-4]_add_|s_quadmask|s_wqm_)")


def scc_violations(asm_lines):
    """(clobbering instruction, reader) pairs: an SCC read whose last SCC
    writer in straight-line order sits inside an inline-asm block
    (;;#ASMSTART .. ;;#ASMEND).  Labels end the scan (no inline sequence
    spans a branch target)."""
    bad, last, in_asm = [], None, False
    for raw in asm_lines:
        line = raw.strip()
        if line.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if line.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if not line or line.startswith(";"):
            continue
        op = line.split()[0]
        if line.endswith(":") or op.startswith("."):
            last = None
            continue
        if SCC_READ.match(op) and last is not None:
            bad.append((last, line))
        if SCC_WRITE.match(op):
            last = line if in_asm else None
    return bad


def test_checker_flags_a_clobbered_branch():
    shift_add = [";;#ASMSTART", "s_lshl1_add_u32 s6, s5, s6", ";;#ASMEND"]
    renorm = [";;#ASMSTART", "s_and_saveexec_b64 s[8:9], s[4:5]", "v_perm_b32 v1, v1, v2, s10",
              "s_mov_b64 exec, s[8:9]", ";;#ASMEND"]
    for seq in (shift_add, renorm):
        assert len(scc_violations(["s_cmp_eq_u32 s4, 1", *seq, "s_cbranch_scc1 .LBB0_2"])) == 1
        assert scc_violations([*seq, "s_cmp_eq_u32 s4, 1", "s_cbranch_scc1 .LBB0_2"]) == []
    # the compiler's own exec narrowing is not an inline sequence
    assert scc_violations(["s_and_saveexec_b64 s[8:9], s[4:5]", "s_cselect_b32 s1, 1, 0"]) == []


@pytest.mark.skipif(shutil.which(_build.HIPCC) is None and not os.path.exists(_build.HIPCC),
                    reason="hipcc not available")
def test_no_scc_read_after_inline_shift_add(tmp_path):
    out = tmp_path / "eq_decode.s"
    flags = [f for f in _build.HIP_FLAGS if f != "-fPIC"]
    subprocess.run([_build.HIPCC, *flags, "--cuda-device-only", "-S",
                    os.path.join(_build.CSRC, "eq_decode.hip"), "-o", str(out)],
                   check=True, capture_output=True)
    lines = out.read_text().splitlines()
    assert sum(1 for ln in lines if ln.strip().startswith("s_lshl1_add_u32")) > 0
    assert sum(1 for ln in lines if ln.strip().startswith("s_and_saveexec_b64")) > 0
    bad = scc_violations(lines)
    assert not bad, f"{len(bad)} SCC reads after the inline shift-add, e.g. {bad[:3]}"
