"""Checks on the gfx950 assembly of the library's own kernels (CPU only).

The gradient kernels (``bwd.hip``) issue their direct-to-LDS ring loads as
inline assembly that sets M0, a register the compiler reserves: clang does not
preserve it around an inline-assembly statement.  That is correct only while
the compiler itself never keeps a value in M0 in those kernels, so the device
assembly of the file is checked here: every M0 write lies inside one of the
inline-assembly statements, and each of those statements is the set-up of one
direct-to-LDS buffer load.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_07713_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
         "-packed-fp32-ops", "--cuda-device-only", "-S", "-Wno-inline-asm"]


def _sources_setting_m0():
    out = []
    for f in sorted(os.listdir(CSRC)):
        if f.endswith((".hip", ".h")):
            text = open(os.path.join(CSRC, f)).read()
            if re.search(r'asm\s+volatile\s*\([^;]*\bm0\b', text, flags=re.S):
                out.append(f)
    return out


def test_only_bwd_sets_m0_in_inline_asm():
    assert _sources_setting_m0() == ["bwd.hip"]


def _m0_writes(asm_text):
    """(inside, outside, blocks): M0 writes inside / outside inline-asm statements, and
    the instruction lists of the statements that write M0."""
    inside, outside, blocks, cur, in_asm = [], [], [], [], False
    for line in asm_text.split("\n"):
        t = line.strip()
        if t.startswith(";;#ASMSTART"):
            in_asm, cur = True, []
            continue
        if t.startswith(";;#ASMEND"):
            if any(re.match(r"\S+\s+m0\s*,", c) for c in cur):
                blocks.append(cur)
            in_asm = False
            continue
        code = t.split(";")[0].strip()
        if not code or code.endswith(":") or code.startswith("."):
            continue
        if in_asm:
            cur.append(code)
        if re.match(r"\S+\s+m0\s*(,|$)", code):
            (inside if in_asm else outside).append(code)
    return inside, outside, blocks


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc missing")
def test_m0_is_written_only_by_the_dma_statements(tmp_path):
    out = str(tmp_path / "bwd.s")
    r = subprocess.run([HIPCC, *FLAGS, os.path.join(CSRC, "bwd.hip"), "-o", out],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    inside, outside, blocks = _m0_writes(open(out).read())
    assert outside == [], f"compiler-generated M0 writes: {outside[:5]}"
    assert inside and len(blocks) == len(inside)
    for b in blocks:
        assert len(b) == 3 and b[0].startswith("s_mov_b32 m0,") and b[1] == "s_nop 0" \
            and b[2].startswith("buffer_load_dwordx4") and b[2].endswith("lds"), b


def test_m0_scan_sees_a_compiler_write():
    # The scan itself: an M0 write outside an inline-assembly statement is reported.
    text = "\n".join([";;#ASMSTART", "s_mov_b32 m0, s4", "s_nop 0",
                      "buffer_load_dwordx4 v1, s[0:3], 0 offen lds", ";;#ASMEND",
                      "s_mov_b32 m0, -1", "ds_read_b32 v0, v1"])
    inside, outside, blocks = _m0_writes(text)
    assert outside == ["s_mov_b32 m0, -1"] and len(inside) == 1 and len(blocks) == 1
