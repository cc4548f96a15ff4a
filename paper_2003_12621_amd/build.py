"""Builds libfftsplit.so in-tree for gfx950 with hipcc.

Usage: python -m paper_2003_12621_amd.build [-v]
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libfftsplit.so")

SOURCES = ["plan.cpp", "api.cpp", "k_weights.hip", "k_forward.hip", "k_contract.hip", "k_inverse.hip", "k_pool.hip",
           "k_direct.hip", "k_oaa.hip", "noalloc.hip", "k_probe.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    # Packed fp32 instructions are kept out of all device code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC] + COMMON + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    if verbose and r.stderr.strip():
        print(r.stderr, file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link libfftsplit.so; returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(16, os.cpu_count() or 1)))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    shutil.move(tmp, LIB)
    return LIB



# Sources each timed kernel is compiled from (for profile-record validity).
KERNEL_SOURCES = {
    "forward": ["k_forward.hip", "band.hpp", "fft_regs.hpp", "twiddles.inc", "launch_util.hpp",
                "fftsplit_internal.hpp"],
    "contract": ["k_contract.hip", "launch_util.hpp", "fftsplit_internal.hpp"],
    "inverse": ["k_inverse.hip", "band.hpp", "fft_regs.hpp", "twiddles.inc", "launch_util.hpp",
                "fftsplit_internal.hpp"],
}


def source_digest(kernel: str = None) -> str:
    """SHA-256 (16 hex digits) over the sources of one kernel, or of the
    whole library when `kernel` is None."""
    import hashlib
    h = hashlib.sha256()
    names = KERNEL_SOURCES[kernel] if kernel else sorted(
        n for n in os.listdir(CSRC) if n.endswith((".hip", ".cpp", ".hpp", ".inc")))
    for name in names:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    if kernel is None:
        with open(os.path.join(ROOT, "include", "fftsplit.h"), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]

if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
