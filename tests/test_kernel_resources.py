"""Static check of the built kernels' register and scratch use.

The hot kernels' speed rests on how many of their workgroups a compute unit
holds at once, and that is set by their LDS and by their vector registers
per lane (a SIMD has 512: 128 registers allow four waves, 168 three, 256
two).  A source change that makes the compiler keep more values live can
silently drop a kernel to fewer resident waves -- a 108-register
contraction kernel at 184 registers ran 20 % slower.  This test reads the
code-object metadata of the built objects (built here from this
repository's sources) and fails if a hot kernel needs more registers than
its occupancy allows, or spills to scratch.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

LLVM = "/opt/rocm/llvm/bin"
BUILD = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2003_12621_amd", "_build")

# (object, kernel-name pattern, largest register count the occupancy allows)
BUDGETS = [
    # three 48 KB workgroups of four waves per CU: three waves per SIMD
    ("k_contract.o", r"contract_kernelILi64ELi64ELi16ELi2ELb1ELi2E", 168),
    ("k_contract.o", r"contract_kernelILi128ELi32ELi16ELi4ELb1ELi2E", 168),
    # 8-channel stages three ahead: four 32 KB workgroups per CU, four waves per SIMD
    ("k_contract.o", r"contract_kernelILi64ELi64ELi8ELi2ELb1ELi3E", 128),
    # four 128-thread workgroups (L = 32) or two 256-thread ones: two waves per SIMD
    ("k_forward.o", r"forward_band_kernelILi32ELi8ELi16E", 256),
    ("k_forward.o", r"forward_band_kernelILi16ELi32ELi8E", 128),
    ("k_inverse.o", r"inverse_band_kernelILi32ELi16ELi16ELb0ELi0E", 256),
    ("k_inverse.o", r"inverse_band_kernelILi16ELi32ELi8ELb0ELi0E", 128),
]


def _metadata(obj, tmp):
    """{kernel symbol: {"vgpr": n, "spill": n}} from the gfx950 code object in obj."""
    fb, co = os.path.join(tmp, "fb.bin"), os.path.join(tmp, "co.o")
    subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fb}", obj,
                    os.path.join(tmp, "copy.o")], check=True, capture_output=True)
    subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o",
                    "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--input={fb}", f"--output={co}"],
                   check=True, capture_output=True)
    r = subprocess.run([f"{LLVM}/llvm-readelf", "--notes", co], check=True, capture_output=True, text=True)
    out, cur = {}, None
    for line in r.stdout.splitlines():
        m = re.match(r"\s*\.name:\s+(\S+)", line)
        if m:
            cur = m.group(1)
            out[cur] = {}
            continue
        m = re.match(r"\s*\.(vgpr_count|vgpr_spill_count):\s+(\d+)", line)
        if m and cur is not None:
            out[cur]["vgpr" if m.group(1) == "vgpr_count" else "spill"] = int(m.group(2))
    return out


@pytest.mark.skipif(not os.path.isdir(BUILD) or not shutil.which(f"{LLVM}/llvm-readelf"),
                    reason="library not built here, or no LLVM tools")
def test_hot_kernels_keep_their_occupancy():
    with tempfile.TemporaryDirectory() as tmp:
        cache = {}
        for obj, pattern, budget in BUDGETS:
            if obj not in cache:
                cache[obj] = _metadata(os.path.join(BUILD, obj), tmp)
            hits = {k: v for k, v in cache[obj].items() if re.search(pattern, k)}
            assert hits, f"{pattern} not found in {obj}"
            for name, res in hits.items():
                assert res.get("spill", 0) == 0, f"{name} spills {res['spill']} registers"
                assert res.get("vgpr", 0) <= budget, f"{name}: {res.get('vgpr')} registers > {budget}"
