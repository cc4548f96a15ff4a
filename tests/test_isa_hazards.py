"""Static check of the built device code for a store-data hazard.

A vector-memory store of more than 8 bytes needs one wait state before a
VALU instruction may overwrite its data registers.  The compiler inserts it
only when the buffer store's scalar offset is not a register; on gfx950 a
16-byte buffer store with a register scalar offset followed at once by a
write of its data registers was measured to store the new value.  The
library therefore passes a constant scalar offset to its 16-byte buffer
stores.  This test disassembles every built object (code objects built here
from this repository's sources) and fails if any store of more than 8 bytes
is immediately followed by a VALU write of one of its data registers.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

LLVM = "/opt/rocm/llvm/bin"
BUILD = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2003_12621_amd", "_build")

STORE = re.compile(r"^\s*(buffer_store_dwordx[34]|global_store_dwordx[34]|flat_store_dwordx[34])\s+v\[(\d+):(\d+)\]")
DEF = re.compile(r"^\s*(v_\w+)\s+v(?:\[(\d+):(\d+)\]|(\d+))\b")


def _regs_written(line):
    m = DEF.match(line)
    if not m or m.group(1).startswith(("v_cmp", "v_readlane", "v_readfirstlane", "v_mfma", "v_accvgpr_write")):
        return set()
    if m.group(4) is not None:
        return {int(m.group(4))}
    return set(range(int(m.group(2)), int(m.group(3)) + 1))


def _disassemble(obj, tmp):
    fb, co = os.path.join(tmp, "fb.bin"), os.path.join(tmp, "co.o")
    # (an explicit output file: without one, llvm-objcopy rewrites its input)
    subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fb}", obj,
                    os.path.join(tmp, "copy.o")], check=True, capture_output=True)
    subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o",
                    "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--input={fb}", f"--output={co}"],
                   check=True, capture_output=True)
    r = subprocess.run([f"{LLVM}/llvm-objdump", "-d", "--mcpu=gfx950", co], check=True, capture_output=True,
                       text=True)
    return [l.split("//")[0] for l in r.stdout.splitlines()]


def hazards(lines):
    found = []
    for i, line in enumerate(lines[:-1]):
        m = STORE.match(line)
        if not m:
            continue
        data = set(range(int(m.group(2)), int(m.group(3)) + 1))
        if _regs_written(lines[i + 1]) & data:
            found.append((line.strip(), lines[i + 1].strip()))
    return found


def test_scanner_finds_the_pattern():
    """The scanner itself, on hand-written lines: a write of a data register
    right after a 16-byte store is flagged; an s_nop in between, an 8-byte
    store, or a write of another register is not."""
    bad = ["\tbuffer_store_dwordx4 v[86:89], v103, s[36:39], s69 offen", "\tv_add_u32_e32 v86, s52, v102"]
    assert len(hazards(bad)) == 1
    assert hazards([bad[0], "\ts_nop 0", bad[1]]) == []
    assert hazards(["\tbuffer_store_dwordx2 v[86:87], v1, s[36:39], s69 offen", bad[1]]) == []
    assert hazards([bad[0], "\tv_add_u32_e32 v90, s52, v102"]) == []


@pytest.mark.skipif(not os.path.isdir(BUILD) or not shutil.which(f"{LLVM}/llvm-objdump"),
                    reason="library not built here, or no LLVM tools")
def test_built_code_has_no_store_data_hazard():
    objs = sorted(os.path.join(BUILD, f) for f in os.listdir(BUILD) if f.startswith("k_") and f.endswith(".o"))
    assert objs, "no kernel objects"
    before = {o: os.stat(o).st_mtime_ns for o in objs}
    with tempfile.TemporaryDirectory() as tmp:
        for obj in objs:
            found = hazards(_disassemble(obj, tmp))
            assert not found, f"{os.path.basename(obj)}: {found[:3]}"
    # the scan reads the build; it must not rewrite it
    assert {o: os.stat(o).st_mtime_ns for o in objs} == before
