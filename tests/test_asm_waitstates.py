"""The hand-counted wait states of the indexer's inline assembly blocks
(MFMA groups and their epilogues) hold in the compiled gfx950 code: the
blocks are found in `hipcc -S` output of index_scores.hip and checked by the
rules stated in `tests/asm_waitstates.py`.  A block with one wait state
taken out of each kind of spacing must be flagged.  CPU only (hipcc
cross-compiles)."""
import os
import shutil
import subprocess

import pytest

from asm_waitstates import blocks, check_block

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SRC = os.path.join(ROOT, "paper_2609_36938_amd", "csrc", "index_scores.hip")

GOOD = """v_mov_b32 v93, 0
s_nop 1
v_mfma_scale_f32_16x16x128_f8f6f4 v[112:115], v[10:17], v[100:107], 0, v90, v90 op_sel:[0,1,0] op_sel_hi:[0,0,0]
v_mfma_scale_f32_16x16x128_f8f6f4 v[116:119], v[2:9], v[100:107], 0, v90, v90 op_sel:[0,1,0] op_sel_hi:[0,0,0]
v_mfma_scale_f32_16x16x128_f8f6f4 v[120:123], v[26:33], v[100:107], 0, v90, v90 op_sel:[0,1,0] op_sel_hi:[0,0,0]
v_mfma_scale_f32_16x16x128_f8f6f4 v[124:127], v[18:25], v[100:107], 0, v90, v90 op_sel:[0,1,0] op_sel_hi:[0,0,0]
s_nop 0
v_cvt_pk_bf16_f32 v112, v112, v113 clamp
v_cvt_pk_bf16_f32 v114, v114, v115 clamp
v_dot2c_f32_bf16 v93, v112, v66
v_cvt_pk_bf16_f32 v116, v116, v117 clamp
v_dot2c_f32_bf16 v93, v114, v67
v_cvt_pk_bf16_f32 v118, v118, v119 clamp
v_dot2c_f32_bf16 v93, v116, v68
v_cvt_pk_bf16_f32 v120, v120, v121 clamp
v_dot2c_f32_bf16 v93, v118, v69
v_cvt_pk_bf16_f32 v122, v122, v123 clamp
v_dot2c_f32_bf16 v93, v120, v70
v_cvt_pk_bf16_f32 v124, v124, v125 clamp
v_dot2c_f32_bf16 v93, v122, v71
v_cvt_pk_bf16_f32 v126, v126, v127 clamp
v_dot2c_f32_bf16 v93, v124, v72
s_nop 0
v_dot2c_f32_bf16 v93, v126, v73
s_nop 2""".splitlines()


# the prefill kernel's group with the head sum on a bf16 MFMA (accumulating form)
GOOD_HS = """s_nop 1
v_mfma_scale_f32_16x16x128_f8f6f4 v[112:115], v[42:49], v[98:105], 0, v96, v96 op_sel:[0,1,0] op_sel_hi:[0,0,0]
v_mfma_scale_f32_16x16x128_f8f6f4 v[116:119], v[34:41], v[98:105], 0, v96, v96 op_sel:[0,1,0] op_sel_hi:[0,0,0]
v_mfma_scale_f32_16x16x128_f8f6f4 v[120:123], v[58:65], v[98:105], 0, v96, v96 op_sel:[0,1,0] op_sel_hi:[0,0,0]
v_mfma_scale_f32_16x16x128_f8f6f4 v[124:127], v[50:57], v[98:105], 0, v96, v96 op_sel:[0,1,0] op_sel_hi:[0,0,0]
s_nop 3
v_cvt_pk_bf16_f32 v112, v112, v113 clamp
v_cvt_pk_bf16_f32 v113, v114, v115 clamp
v_cvt_pk_bf16_f32 v114, v116, v117 clamp
v_cvt_pk_bf16_f32 v115, v118, v119 clamp
v_cvt_pk_bf16_f32 v116, v120, v121 clamp
v_cvt_pk_bf16_f32 v117, v122, v123 clamp
s_nop 1
v_cvt_pk_bf16_f32 v118, v124, v125 clamp
v_cvt_pk_bf16_f32 v119, v126, v127 clamp
s_nop 1
v_mfma_f32_16x16x32_bf16 v[82:85], v[74:77], v[112:115], v[82:85]
v_mfma_f32_16x16x32_bf16 v[82:85], v[78:81], v[116:119], v[82:85]
s_nop 7""".splitlines()


def test_rules_accept_the_documented_group():
    assert check_block(GOOD) == []
    assert check_block(GOOD_HS) == []


@pytest.mark.parametrize("old,new,expect", [
    ("s_nop 3", "s_nop 2", "12"),                                        # converts read the last MFMAs early
    ("v_cvt_pk_bf16_f32 v119, v126, v127 clamp\ns_nop 1", "v_cvt_pk_bf16_f32 v119, v126, v127 clamp",
     "(< 2)"),                                                           # MFMA reads a fresh convert
    ("\ns_nop 7", "", "4-pass MFMA"),                                    # head sum read right after the block
    ("v[116:119], v[82:85]", "v[116:119], v[83:86]", "(< 8)"),           # not an exact accumulation
])
def test_rules_flag_the_head_sum_group(old, new, expect):
    text = "\n".join(GOOD_HS)
    assert old in text
    bad = check_block(text.replace(old, new, 1).splitlines())
    assert any(expect in v for v in bad), bad


@pytest.mark.parametrize("drop,expect", [
    ("s_nop 0\nv_cvt_pk_bf16_f32 v112", "12"),   # MFMA result read one wait state early
    ("s_nop 2", "block end"),                     # dot result left 0 wait states before the block ends
    ("s_nop 1\nv_mfma", "first MFMA"),            # no room after a VALU write of an MFMA source
])
def test_rules_flag_a_missing_wait_state(drop, expect):
    text = "\n".join(GOOD)
    first, _, rest = drop.partition("\n")
    i = text.index(drop)
    bad = (text[:i] + rest + text[i + len(drop):]).splitlines()
    assert any(expect in v for v in check_block(bad)), check_block(bad)


def test_rules_flag_a_convert_read_at_once():
    bad = [l for l in GOOD]
    # the dot that reads v114 straight after its convert
    j = bad.index("v_dot2c_f32_bf16 v93, v112, v66")
    bad[j] = "v_dot2c_f32_bf16 v93, v114, v66"
    assert any("v114" in v for v in check_block(bad))


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc not installed")
def test_compiled_indexer_blocks(tmp_path):
    out = tmp_path / "index_scores.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-I" + os.path.join(ROOT, "include"), "-I" + os.path.dirname(SRC),
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", SRC, "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    bl = [b for b in blocks(out.read_text()) if any(l.startswith("v_mfma") for l in b)]
    # fp8 groups (prefill with bf16 head sums, and row kernels), the widened
    # MXFP4 group, and the MXFP4 prefill group with fp4 B operands
    assert len(bl) >= 4
    assert any("blgp:4" in l for b in bl for l in b)
    assert any("v_mfma_f32_16x16x32_bf16" in l for b in bl for l in b)
    bad = [v for b in bl for v in check_block(b)]
    assert not bad, "\n".join(bad[:20])
