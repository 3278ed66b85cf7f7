"""Checks on the gfx950 assembly of the library's own kernels (CPU only).

A clamp of a 64-bit uniform value, min(SLOT, e - t0), was once lowered to a
vector compare followed by a scalar select that read the scalar condition
code after an unrelated add had overwritten it, so the clamp took the wrong
value.  The kernels now clamp in 32 bits; this test compiles the device code
to assembly and fails if any value-selecting s_cselect reads a condition code
last written by a carry-producing add or subtract.
"""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2304_00737_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

CARRY_WRITERS = ("s_add_u32", "s_addc_u32", "s_sub_u32", "s_subb_u32")
SCC_WRITER = re.compile(
    r"^\s*(s_cmp\w*|s_cmpk\w*|s_add_u32|s_addc_u32|s_sub_u32|s_subb_u32|s_add_i32|s_sub_i32|s_addk\w*|"
    r"s_and_\w+|s_or_\w+|s_xor_\w+|s_andn2\w*|s_orn2\w*|s_nand\w*|s_nor\w*|s_xnor\w*|s_lshl\w*|s_lshr\w*|"
    r"s_ashr\w*|s_bfe\w*|s_min\w*|s_max\w*|s_abs\w*|s_not\w*|s_bcnt\w*|s_ff\w*|s_bitcmp\w*)\b")


def suspicious_selects(asm: str):
    lines = asm.splitlines()
    out, fn = [], None
    for i, line in enumerate(lines):
        m = re.match(r"^(_Z\w+):", line)
        if m:
            fn = m.group(1)
        if not re.match(r"^\s*s_cselect", line) or re.search(r",\s*-1,\s*0\s*$", line):
            continue
        for j in range(i - 1, max(i - 80, -1), -1):
            t = lines[j]
            if re.match(r"^[^\s;].*:", t):
                break
            w = SCC_WRITER.match(t)
            if w:
                if w.group(1) in CARRY_WRITERS:
                    out.append(f"{fn}: {line.strip()} <- {t.strip()}")
                break
    return out


KERNEL_FILES = ["kernels_add.hip", "kernels_select.hip", "kernels_merge.hip", "kernels_decode.hip",
                "kernels_variants.hip"]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
@pytest.mark.parametrize("src", KERNEL_FILES)
def test_no_select_reads_a_carry(tmp_path, src):
    asm = tmp_path / (src + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-ffp-contract=off",
           "-fno-gpu-flush-denormals-to-zero", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", str(asm)]
    subprocess.run(cmd, check=True, capture_output=True, timeout=600)
    bad = suspicious_selects(asm.read_text())
    assert not bad, "\n".join(bad[:10])


def test_every_kernel_file_is_checked():
    from paper_2304_00737_amd import build
    assert sorted(KERNEL_FILES) == sorted(f for f in build.KERNEL_SOURCES if f != "api.hip")


def test_detector_flags_the_known_pattern():
    asm = "\n".join([
        "_Zkernel:",
        "\tv_cmp_lt_i64_e32 vcc, s[0:1], v[2:3]",
        "\ts_addc_u32 s41, s19, s3",
        "\ts_cbranch_vccz .LBB0_1",
        "; %bb.1:",
        "\ts_cselect_b32 s47, s0, 0x1000",
        "\ts_cmpk_lt_u32 s55, 0x1000",
        "\ts_cselect_b32 s5, s55, s6",
        "\ts_add_u32 s1, s2, s3",
        "\ts_cselect_b64 s[4:5], -1, 0",
    ])
    bad = suspicious_selects(asm)
    assert len(bad) == 1 and "s47" in bad[0]
