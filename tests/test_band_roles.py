"""Host check of the patch-pair lane roles of the band transforms
(PairRole in csrc/band.hpp): compiled with hipcc for the host and run on
the CPU.  For every work-item size that uses them, the roles cover each
(patch, column) of an item exactly once; lanes l and l + 32 of a wave hold
patches 2m and 2m + 1 of one column (what one 16-byte access of two
consecutive patches and a half-wave exchange need); and each 16
consecutive lanes' 8-byte LDS accesses of one half-spectrum row
(patch * stride + column, stride = band_half_stride) fall in 16 distinct
bank pairs."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2003_12621_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"

SRC = r"""
#include <cstdio>
#include "band.hpp"
#include "fftsplit_internal.hpp"
using namespace fftsplit;

template <int L, int TG>
static int check() {
    constexpr int H2 = L / 2, NT = TG * H2, TTS = band_half_stride(L, TG);
    int seen[TG][H2] = {};
    int bad = 0;
    for (int wv = 0; wv < NT / 64; ++wv) {
        for (int l = 0; l < 64; ++l) {
            const PairRole<TG> r(l, wv);
            if (r.patch < 0 || r.patch >= TG || r.col < 0 || r.col >= H2) { ++bad; continue; }
            ++seen[r.patch][r.col];
            if (l < 32) {
                const PairRole<TG> u(l + 32, wv);
                if (u.pm != r.pm || u.col != r.col || r.patch != 2 * r.pm || u.patch != 2 * r.pm + 1) ++bad;
            }
        }
        for (int g = 0; g < 64; g += 16) {
            int used[16] = {};
            for (int l = g; l < g + 16; ++l) {
                const PairRole<TG> r(l, wv);
                ++used[(r.patch * TTS + r.col) % 16];
            }
            for (int b = 0; b < 16; ++b) bad += used[b] != 1;
        }
    }
    for (int p = 0; p < TG; ++p)
        for (int c = 0; c < H2; ++c) bad += seen[p][c] != 1;
    std::printf("L=%d TG=%d stride=%d bad=%d\n", L, TG, TTS, bad);
    return bad;
}

int main() { return (check<32, 16>() + check<16, 32>() + check<32, 8>()) ? 1 : 0; }
"""


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_pair_roles(tmp_path):
    src = tmp_path / "roles.hip"
    src.write_text(SRC)
    exe = tmp_path / "roles"
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-std=c++17", "-I", CSRC, "-I", os.path.join(ROOT, "include"),
                    str(src), "-o", str(exe)], check=True, capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    print(r.stdout)
    assert r.returncode == 0, r.stdout
    assert r.stdout.count("bad=0") == 3
