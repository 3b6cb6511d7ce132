"""Static checks of the gfx950 device assembly the library's kernels compile to
(CPU only: hipcc emits the assembly, nothing runs on a GPU).

DPP wait states.  On gfx950 a DPP instruction that reads a VGPR written by a
VALU instruction needs two wait states between them.  The compiler inserts
them for the DPP instructions it emits itself, but not for DPP moves written
as inline assembly (the lane-pair contraction's partner moves), which must
carry their own s_nop.  A missing wait state makes the move read the old
register value: a wrong partner value for one product, no fault, and an
error that only some outputs show.  The scan walks every kernel's
instruction stream and checks each DPP read against the VALU writes of the
two wait states before it.
"""

import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2509_24093_amd")
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
HIPCC = "/opt/rocm/bin/hipcc"

pytestmark = pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")

_REG = re.compile(r"^v(\d+)$|^v\[(\d+):(\d+)\]$")


def _vgprs(op):
    m = _REG.match(op.strip())
    if not m:
        return set()
    if m.group(1) is not None:
        return {int(m.group(1))}
    return set(range(int(m.group(2)), int(m.group(3)) + 1))


def dpp_hazards(asm_text):
    """(write, dpp) instruction pairs where a DPP instruction reads the VGPR
    (its first source operand) that a VALU instruction wrote fewer than two
    wait states before.  Labels end the look-back (a branch target has other
    predecessors, which the scan does not follow)."""
    instrs = []
    for line in asm_text.splitlines():
        t = line.split(";")[0].strip()
        if not t or t.startswith("."):
            continue
        if t.endswith(":"):
            instrs.append(None)
            continue
        instrs.append(t)
    found = []
    for n, t in enumerate(instrs):
        if t is None or not ("_dpp" in t or "quad_perm:" in t or "row_" in t.split(" ", 1)[-1]):
            continue
        ops = [o for o in t.split(None, 1)[1].split(",")] if " " in t else []
        if len(ops) < 2:
            continue
        src = _vgprs(ops[1].split()[0])
        ws = 0
        for j in range(n - 1, -1, -1):
            pt = instrs[j]
            if pt is None or ws >= 2:
                break
            if pt.startswith("s_nop"):
                ws += int(pt.split()[1], 0) + 1
                continue
            if pt.startswith("v_"):
                dst = _vgprs(pt.split(None, 1)[1].split(",")[0]) if " " in pt else set()
                if dst & src:
                    found.append((pt, t))
                    break
            ws += 1
    return found


def test_scanner_sees_a_hazard_and_its_fix():
    bad = "v_fmac_f32_e32 v106, 0x3cbcf890, v8\nv_mov_b32_dpp v2, v106 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n"
    one = "v_add_f32_e32 v106, v1, v2\nv_mul_f32_e32 v7, v1, v2\nv_mov_b32_dpp v2, v106 quad_perm:[1,0,3,2]\n"
    ok = "v_fmac_f32_e32 v106, 0x3cbcf890, v8\ns_nop 1\nv_mov_b32_dpp v2, v106 quad_perm:[1,0,3,2] row_mask:0xf\n"
    far = "v_add_f32_e32 v106, v1, v2\nv_mul_f32_e32 v7, v1, v2\nv_mul_f32_e32 v8, v1, v2\nv_mov_b32_dpp v2, v106 quad_perm:[1,0,3,2]\n"
    wide = "v_lshlrev_b64 v[106:107], 1, v[0:1]\nv_mov_b32_dpp v2, v107 quad_perm:[1,0,3,2]\n"
    assert len(dpp_hazards(bad)) == 1
    assert len(dpp_hazards(one)) == 1
    assert dpp_hazards(ok) == []
    assert dpp_hazards(far) == []
    assert len(dpp_hazards(wide)) == 1


@pytest.fixture(scope="module")
def gen_dir(tmp_path_factory):
    d = tmp_path_factory.mktemp("gen")
    gen = str(d / "gen_cg")
    subprocess.run(["g++", "-O2", "-std=c++17", os.path.join(CSRC, "codegen", "gen_cg.cpp"),
                    os.path.join(CSRC, "cg_table.cpp"), "-o", gen], check=True, capture_output=True)
    subprocess.run([gen, str(d), "8"], check=True, capture_output=True)
    return d


# kernels with DPP moves: the lane-pair contraction (L_max 7; 8 is the same
# code), the fused kernel's channel-pair stores, the inter-channel kernel, the
# lane-pair channel-mixing kernel and the one-block kernel for short token axes
UNITS = [("cg_gen.hip", 7), ("cg_fused.hip", 6), ("cg_inter.hip", 4), ("cg_mix.hip", 3), ("cg_small.hip", 3)]


@pytest.mark.parametrize("unit", UNITS, ids=lambda u: "%s-L%d" % u)
def test_no_dpp_read_within_two_wait_states_of_its_write(unit, gen_dir, tmp_path):
    src, L = unit
    out = str(tmp_path / "k.s")
    cmd = [HIPCC, "-S", "--offload-device-only", "--offload-arch=gfx950", "-O3", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + str(gen_dir), "-I" + CSRC, "-I" + INCLUDE,
           "-DCGCONV_TU_L=%d" % L, '-DCGCONV_BODY="cg_body_L%d.inc"' % L, os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    text = open(out).read()
    n_dpp = sum(1 for l in text.splitlines() if "quad_perm:" in l or "_dpp " in l)
    assert n_dpp > 0, "no DPP instruction found: the scan would check nothing"
    bad = dpp_hazards(text)
    assert not bad, "%d DPP reads too close to their VALU write, e.g. %r" % (len(bad), bad[:3])
