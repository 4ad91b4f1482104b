"""The grouped GEMM's direct-to-LDS loads are an inline-assembly statement that sets M0
with a scalar add, which also writes SCC.  If the compiler held a compare result, or the
carry of a 64-bit address add split in two, in SCC across that statement, the branch or
the high half of the address would read the statement's SCC instead (a wrong branch, or
an address 4 GiB off whenever the low half carries).  The statement declares SCC
clobbered; this test compiles the sources that instantiate the GEMMs to gfx950 assembly
and checks that no instruction reads SCC after the statement before something writes
it again.  CPU only (the compiler cross-compiles)."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2002_04013_amd import build as B

HIPCC = B.HIPCC
SOURCES = ["ffn.hip", "ffblock.hip"]

# scalar instructions that read SCC
READERS = re.compile(r"^(s_cbranch_scc[01]|s_cselect_b(32|64)|s_addc_u32|s_subb_u32|s_cmov_b(32|64)|s_cmovk_i32)\b")
# scalar instructions that neither read nor write SCC
NEUTRAL = re.compile(r"^(s_mov_|s_movk_|s_nop|s_waitcnt|s_barrier|s_setprio|s_sleep|s_load|s_buffer_load|"
                     r"s_getpc|s_branch|s_cbranch_exec|s_cbranch_vcc|s_sched|s_dcache|s_icache|s_getreg|"
                     r"s_setreg|s_memtime|s_memrealtime|s_sendmsg)")


def scc_hazards(asm_lines):
    """(line of the m0 add, line of the reader) for every SCC reader reached from an
    inline-assembly 'S_ADD_U32 m0' before any SCC writer or label."""
    lines = [l.split(";")[0].strip() for l in asm_lines]
    bad = []
    for i, l in enumerate(lines):
        if not l.startswith("s_add_u32 m0"):
            continue
        for j in range(i + 1, min(i + 400, len(lines))):
            t = lines[j]
            if not t or t.startswith("."):
                if t.endswith(":"):
                    break                       # a label: another path may join here
                continue
            if t.endswith(":"):
                break
            op = t.split()[0]
            if READERS.match(op):
                bad.append((i + 1, j + 1))
                break
            if op.startswith("s_") and not NEUTRAL.match(op):
                break                           # an SCC writer: the statement's SCC is dead
    return bad


def test_scanner_flags_a_carry_split_around_the_load():
    """The scan itself: a carry split around the statement is flagged, a re-written SCC is not."""
    split = ["s_add_u32 s46, s40, 0x180", "s_add_u32 m0, s50, 0", "s_nop 0",
             "global_load_lds_dwordx4 v4, s[48:49]", "s_addc_u32 s47, s41, 0"]
    assert scc_hazards(split) == [(2, 5)]
    rewritten = ["s_cmp_lt_u32 s3, 64", "s_add_u32 m0, s50, 0", "global_load_lds_dwordx4 v4, s[48:49]",
                 "s_cmp_lt_u32 s3, 64", "s_cbranch_scc1 .LBB0_1"]
    assert scc_hazards(rewritten) == []


@pytest.mark.skipif(not (os.path.exists(HIPCC) or shutil.which("hipcc")), reason="hipcc not installed")
@pytest.mark.parametrize("src", SOURCES)
def test_no_scc_reader_after_direct_lds_load(src, tmp_path):
    out = tmp_path / (src + ".s")
    cmd = [HIPCC, *B.CFLAGS, "--cuda-device-only", "-S", os.path.join(B.CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(out) as f:
        lines = f.readlines()
    assert any("global_load_lds_dwordx4" in l for l in lines), "no direct-to-LDS load compiled"
    bad = scc_hazards(lines)
    assert not bad, f"SCC read after the direct-to-LDS statement at assembly lines {bad[:5]}"
