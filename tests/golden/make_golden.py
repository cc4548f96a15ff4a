"""Writes the stored expected values under tests/golden/.

It calls only the oracle package.  Run from the repository root:
    python tests/golden/make_golden.py
"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import opcount  # noqa: E402


def write_opcounts(path):
    lines = ["# Operation counts of Section 3.2, eqs. (11)-(14), per channel pair.",
             "# columns: function image_size kernel patch(0 = none) value",
             "# written by tests/golden/make_golden.py from oracle.opcount"]
    for n in (32, 56, 224):
        for k in (3, 5):
            lines.append(f"mul_oaaconv {n} {k} 0 {opcount.mul_oaaconv(n, k)!r}")
            lines.append(f"add_oaaconv {n} {k} 0 {opcount.add_oaaconv(n, k)!r}")
            for s in (6, 16, 32):
                lines.append(f"mul_splitconv {n} {k} {s} {opcount.mul_splitconv(n, k, s)!r}")
                lines.append(f"add_splitconv {n} {k} {s} {opcount.add_splitconv(n, k, s)!r}")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def write_fig3(path, n=224):
    """Fig. 3's comparison as numbers: total operations (#MUL + #ADD) per
    channel pair of an n x n image against the kernel size, for SplitConv
    with patch sizes s = 16 and 32 (eqs. 13-14) and for OaAConv (eqs.
    11-12).  The figure prints no values and names no image size; every
    count scales with n^2, so the ratios do not depend on it."""
    lines = ["# Section 3.2, Fig. 3: #MUL + #ADD per channel pair of a "
             f"{n}x{n} image (eqs. 11-14)",
             "# columns: k oaaconv split_s16 split_s32 oaaconv/split_s16 oaaconv/split_s32",
             "# written by tests/golden/make_golden.py from oracle.opcount"]
    for k in range(3, 12, 2):
        oaa = opcount.mul_oaaconv(n, k) + opcount.add_oaaconv(n, k)
        s16 = opcount.mul_splitconv(n, k, 16) + opcount.add_splitconv(n, k, 16)
        s32 = opcount.mul_splitconv(n, k, 32) + opcount.add_splitconv(n, k, 32)
        lines.append(f"{k} {oaa!r} {s16!r} {s32!r} {oaa / s16!r} {oaa / s32!r}")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    write_opcounts(os.path.join(HERE, "opcounts.txt"))
    write_fig3(os.path.join(HERE, "fig3_opcounts.txt"))
