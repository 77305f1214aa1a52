"""Wide vector-memory stores keep their data registers intact until the
hardware has read them.

A 16-byte (or 12-byte) store reads its data VGPRs after it issues; the
instruction right behind it must not overwrite them.  The compiler inserts the
wait state for that except when a buffer store's SGPR offset is a register, and
on gfx950 such a store was seen writing the next instruction's result instead
of its data.  This test compiles the kernels to gfx950 assembly, as the
library build does, and checks that (1) no wide buffer store takes a register
SGPR offset and (2) no wide store is followed directly by a VALU instruction
writing one of its data registers.  It needs hipcc (not a GPU).
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2609_26219_amd import build as pkv_build

WIDE_STORE = re.compile(r"^(buffer|global|flat|scratch)_store_(dwordx3|dwordx4|b96|b128|format_xyzw?)\b")


def _vgprs(tok: str) -> set:
    m = re.match(r"v\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def scan(asm: str) -> tuple:
    """(problems found in one assembly listing, number of wide stores in it)."""
    lines = [l.strip() for l in asm.splitlines()]
    code = [l for l in lines if l and not l.startswith((";", ".")) and not l.endswith(":")]
    problems, n_wide = [], 0
    for i, ins in enumerate(code):
        m = WIDE_STORE.match(ins)
        if not m:
            continue
        n_wide += 1
        ops = [o.strip() for o in ins.split(None, 1)[1].split(",")]
        data = _vgprs(ops[0] if m.group(1) == "buffer" else ops[1])
        if m.group(1) == "buffer" and re.match(r"s\d+$|s\[", ops[3].split()[0]):
            problems.append(f"register SGPR offset: {ins}")
        nxt = code[i + 1] if i + 1 < len(code) else ""
        if nxt.startswith("v_") and not nxt.startswith(("v_cmp", "v_readlane", "v_readfirstlane")):
            dst = nxt.split(None, 1)[1].split(",")[0].strip() if " " in nxt else ""
            if _vgprs(dst) & data:
                problems.append(f"data register rewritten right after the store: {ins} / {nxt}")
    return problems, n_wide


def test_scanner_flags_both_patterns():
    bad = "\n".join([
        "buffer_store_dwordx4 v[0:3], v8, s[48:51], s10 offen nt",
        "v_add_u32_e32 v0, v48, v68",
    ])
    found, n = scan(bad)
    assert n == 1
    assert any("register SGPR offset" in p for p in found)
    assert any("rewritten" in p for p in found)
    good = "\n".join([
        "buffer_store_dwordx4 v[0:3], v8, s[48:51], 0 offen nt",
        "s_nop 0",
        "v_add_u32_e32 v0, v48, v68",
        "buffer_store_dwordx2 v[4:5], v9, s[48:51], s10 offen",
        "v_mov_b32_e32 v4, 0",
    ])
    assert scan(good) == ([], 1)


@pytest.mark.skipif(not os.path.exists(pkv_build.HIPCC) and shutil.which("hipcc") is None, reason="needs hipcc")
@pytest.mark.parametrize("src", ["restore.hip", "gather.hip"])
def test_kernels_have_no_store_data_hazard(src, tmp_path):
    out = tmp_path / (src + ".s")
    cmd = [pkv_build.HIPCC, *pkv_build.HIP_FLAGS, "--cuda-device-only", "-S",
           os.path.join(pkv_build.CSRC, src), "-o", str(out)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    problems, n_wide = scan(out.read_text())
    assert n_wide > 0  # the kernels write 16-byte pieces
    assert not problems, "\n".join(problems[:10])
