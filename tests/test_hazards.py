"""The generated-code hazard check that the build runs (paper_2609_07108_amd
/hazards.py), on hand-written gfx950 assembly: each rule is shown to catch a
violation and to accept the padded form, including across a branch."""

from paper_2609_07108_amd import hazards as Hz


def _fn(body: str) -> str:
    return ("\t.type\tk,@function\nk:\n" + "\n".join("\t" + l if not l.endswith(":") else l
                                                   for l in body.strip().splitlines()) + "\n.Lfunc_end0:\n")


def _rules(body):
    return sorted({e.split(": ")[1].split()[0] for e in Hz.check_asm(_fn(body))})


MFMA = "v_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], v[20:23], v[0:15]"


def test_r1_mfma_result_read_too_early():
    assert _rules(f"{MFMA}\nv_add_f32_e32 v30, v31, v32\nv_mul_f32_e32 v33, v5, v5\ns_endpgm") == ["R1"]


def test_r1_padded_read_and_accumulation_chain_are_fine():
    assert _rules(f"{MFMA}\n{MFMA}\ns_nop 15\nv_mul_f32_e32 v33, v5, v5\ns_endpgm") == []


def test_r1_result_used_as_operand_or_overwritten():
    assert _rules(f"{MFMA}\nv_mfma_f32_32x32x16_bf16 v[32:47], v[0:3], v[20:23], 0\ns_nop 15\ns_endpgm") == ["R1"]
    assert _rules(f"{MFMA}\nds_read_b128 v[4:7], v40\ns_nop 15\ns_endpgm") == ["R1"]
    assert _rules(f"{MFMA}\nv_accvgpr_write_b32 a0, v3\ns_nop 15\ns_endpgm") == ["R1"]


def test_r1_follows_branches():
    body = f"""
{MFMA}
s_cbranch_scc1 .LBB0_2
s_nop 15
s_endpgm
.LBB0_2:
v_mov_b32_e32 v40, v7
s_endpgm
"""
    assert _rules(body) == ["R1"]


def test_r2_valu_write_then_inline_mfma():
    bad = """
v_cvt_pk_bf16_f32 v17, v40, v41
;;#ASMSTART
v_mfma_f32_32x32x16_bf16 a[0:15], v[16:19], v[20:23], a[0:15]
;;#ASMEND
s_endpgm
"""
    assert _rules(bad) == ["R2"]
    good = bad.replace(";;#ASMSTART\n", ";;#ASMSTART\ns_nop 1\n")
    assert _rules(good) == []


def test_r3_m0_then_direct_load():
    bad = "s_mov_b32 m0, s6\nglobal_load_lds_dwordx4 v2, s[26:27]\ns_endpgm"
    assert _rules(bad) == ["R3"]
    assert _rules(bad.replace("\nglobal", "\ns_nop 0\nglobal")) == []
