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


if __name__ == "__main__":
    write_opcounts(os.path.join(HERE, "opcounts.txt"))
