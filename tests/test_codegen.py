"""Static checks on the gfx950 assembly of the HIP sources (CPU only).

The kernels issue their HBM -> LDS tile copies from inline assembly that sets
m0 and adds with s_add_u32, which writes the scalar carry bit (SCC).  A
compiler 64-bit scalar add is an s_add_u32 / s_addc_u32 pair that passes its
carry through SCC, so no SCC-writing instruction, and no inline assembly, may
sit between the two halves: a lost carry puts the high address word 4 GiB off.
These tests compile every source to assembly with the library's own flags and
check that property, that m0 is written only by that inline assembly, and two
hardware rules the kernels follow: no scalar-cache stores or atomics and no
packed fp32 VALU instructions.
"""
from __future__ import annotations

import os
import re
import subprocess

import pytest

from paper_2608_02504_amd import build as B

HIP_SOURCES = [s for s in B.sources() if s.endswith(".hip")]

# SALU opcodes that write SCC (gfx9 encoding families); s_addc_u32 itself reads it
SCC_WRITERS = re.compile(
    r"^s_(add|addc|sub|subb|min|max|and|or|xor|andn2|orn2|nand|nor|xnor|lshl|lshr|ashr|"
    r"bfe|bcnt|abs|not|cmp|bitcmp|addk|cmpk|mulk|lshl\d_add|absdiff|quadmask|wqm)[_a-z0-9]*\b"
)


def _have_hipcc() -> bool:
    try:
        B.hipcc()
        return True
    except RuntimeError:
        return False


pytestmark = pytest.mark.skipif(not _have_hipcc(), reason="hipcc not available")


@pytest.fixture(scope="module")
def assembly(tmp_path_factory):
    out = {}
    d = tmp_path_factory.mktemp("asm")
    for src in HIP_SOURCES:
        dst = os.path.join(d, os.path.basename(src) + ".s")
        cmd = [B.hipcc(), *B.COMMON, "--cuda-device-only", "-S", src, "-o", dst]
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-2000:]
        out[os.path.basename(src)] = open(dst).read()
    return out


def _kernels(text: str):
    """(name, [instruction or marker lines]) per kernel; markers are ASMSTART/ASMEND."""
    for m in re.finditer(r"\n(_Z\S+):[^\n]*\n", text):
        body = text[m.end():]
        end = body.find("s_endpgm")
        body = body[: end if end >= 0 else len(body)]
        lines = []
        for ln in body.splitlines():
            t = ln.strip()
            if t.startswith(";;#ASMSTART"):
                lines.append("ASMSTART")
            elif t.startswith(";;#ASMEND"):
                lines.append("ASMEND")
            elif t and not t.startswith((";", ".")):
                lines.append(t)
        yield m.group(1), lines


def test_sources_found():
    assert any(s.endswith("attn_bf16.hip") for s in HIP_SOURCES)


SCC_READERS = re.compile(r"^(s_addc_u32|s_subb_u32|s_cselect_|s_cbranch_scc|s_cmov_|s_cmovk_)")


def test_inline_asm_does_not_clobber_live_scc(assembly):
    """After every inline-asm block that writes SCC, the next instruction that
    touches SCC must write it, not read it: a read would consume the value the
    asm destroyed (e.g. the carry between the halves of a 64-bit add)."""
    checked = 0
    for fname, text in assembly.items():
        for kname, lines in _kernels(text):
            i = 0
            while i < len(lines):
                if lines[i] != "ASMSTART":
                    i += 1
                    continue
                j = lines.index("ASMEND", i)
                block = lines[i + 1:j]
                i = j + 1
                if not any(SCC_WRITERS.match(t) for t in block):
                    continue
                checked += 1
                for u in lines[j + 1:]:
                    if u in ("ASMSTART", "ASMEND"):
                        continue
                    assert not SCC_READERS.match(u), \
                        f"{fname}:{kname}: '{u}' reads SCC clobbered by inline asm {block}"
                    if SCC_WRITERS.match(u) or u.startswith(("s_branch", "s_endpgm", "s_setpc")):
                        break
    assert checked > 0


def test_m0_written_only_by_tile_copy_asm(assembly):
    for fname, text in assembly.items():
        for kname, lines in _kernels(text):
            in_asm = False
            for t in lines:
                if t in ("ASMSTART", "ASMEND"):
                    in_asm = t == "ASMSTART"
                    continue
                if not in_asm:
                    ops = t.split(None, 1)
                    assert not (len(ops) > 1 and re.search(r"\bm0\b", ops[1])), \
                        f"{fname}:{kname}: compiler-generated use of m0: '{t}'"


def test_no_scalar_stores_or_packed_fp32(assembly):
    banned = re.compile(r"^(s_store|s_buffer_store|s_scratch_store|s_atomic|s_buffer_atomic|"
                        r"s_dcache_wb|s_dcache_discard|v_pk_add_f32|v_pk_mul_f32|v_pk_fma_f32)")
    for fname, text in assembly.items():
        for kname, lines in _kernels(text):
            for t in lines:
                assert not banned.match(t), f"{fname}:{kname}: '{t}'"
