"""The LDA sampler's DPP reads keep the wait states the hardware needs (no GPU).

On CDNA a DPP instruction must not read a VGPR that a VALU instruction wrote in the two
wait states before it (each instruction is one wait state, s_nop n is n + 1).  The sampler's
hand-written DPP steps (the 64-bit prefix scan and the exponent maximum) carry their own
s_nop where nothing else can fill the gap, and the exponent maximum relies on the Newton
steps that scheduling barriers pin between its steps.  The compiler sees neither inside the
inline assembly, so this test compiles the sampler for gfx950 and checks every DPP read of
the generated code.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCE = os.path.join(ROOT, "paper_1410_8043_amd", "csrc", "ps_lda.hip")

# VALU instructions whose first operand is not a VGPR they write
NO_VGPR_DEST = ("v_cmp", "v_cmpx", "v_readlane", "v_readfirstlane")


def vgprs(operand):
    m = re.fullmatch(r"v(\d+)", operand)
    if m:
        return {int(m.group(1))}
    m = re.fullmatch(r"v\[(\d+):(\d+)\]", operand)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    return set()


def parse(asm_text):
    """(mnemonic, operands) per instruction, None at labels and function boundaries."""
    out = []
    for raw in asm_text.splitlines():
        line = raw.split(";")[0].strip()
        if not line:
            continue
        if line.endswith(":") or line.startswith(".end_amdhsa_kernel") or line.startswith(".Lfunc_end"):
            out.append(None)
            continue
        if line.startswith("."):
            continue
        parts = line.split(None, 1)
        ops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
        out.append((parts[0], ops))
    return out


def dpp_hazards(instrs):
    """Every DPP read whose operand a VALU instruction wrote less than two wait states before."""
    bad, checked = [], 0
    for i, ins in enumerate(instrs):
        if ins is None or not ins[0].endswith("_dpp"):
            continue
        name, ops = ins
        src = ops[2] if name.startswith(("v_add_co_u32", "v_addc_co_u32", "v_sub_co_u32", "v_subb_co_u32")) else ops[1]
        read = vgprs(src)
        assert read, (name, ops)
        waits, j = 0, i - 1
        while waits < 2:
            prev = instrs[j]
            if prev is None:  # a label: the code before it need not be what runs before
                bad.append((i, name, "label within two wait states"))
                break
            pname, pops = prev
            if pname == "s_nop":
                waits += int(pops[0], 0) + 1
            else:
                if pname.startswith("v_") and not pname.startswith(NO_VGPR_DEST) and pops and vgprs(pops[0]) & read:
                    bad.append((i, name, f"{pname} {', '.join(pops)} after {waits} wait states"))
                    break
                waits += 1
            j -= 1
        checked += 1
    return bad, checked


def test_every_dpp_read_of_the_sampler_has_two_wait_states(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not found")
    out = tmp_path / "ps_lda.s"
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
                    "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-S", SOURCE,
                    "-o", str(out)], check=True, capture_output=True)
    text = out.read_text()
    bad, checked = dpp_hazards(parse(text))
    # 12 scan and 6 maximum steps in every instantiation of the sampling kernel
    assert checked >= 18 * len(re.findall(r"^_ZN\S*k_lda_sweep\S*:", text, re.M))
    assert not bad, bad[:5]


def test_the_checker_finds_a_missing_wait():
    # a planted hazard: the DPP step right after the write of its operand, then after one
    # instruction, then with enough wait states
    asm = """
    v_add_u32_e32 v12, 1, v12
    v_max_i32_dpp v12, v12, v12 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf
    v_fma_f64 v[4:5], v[6:7], v[8:9], 1.0
    v_max_i32_dpp v12, v12, v12 row_mirror row_mask:0xf bank_mask:0xf
    s_nop 0
    v_mov_b32_e32 v3, v12
    v_max_i32_dpp v12, v12, v12 row_half_mirror row_mask:0xf bank_mask:0xf
    s_nop 1
    v_add_co_u32_dpp v14, vcc, v14, v14 row_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1
    """
    bad, checked = dpp_hazards(parse(asm))
    assert checked == 4
    assert [b[0] for b in bad] == [1, 3]
