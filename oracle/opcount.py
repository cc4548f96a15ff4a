"""Operation counts of Section 3.2, eqs. (11)-(14) (test infrastructure only).

Counts are per (input channel, output channel) pair over an N x N image with
a k x k kernel.  The printed "log(2k-1)^2" and "log(s+k-1)^2" are read as the
base-2 logarithm of the squared FFT size (the 2-D point count), which is the
Cooley-Tukey stage count of a radix-2 2-D transform.
"""
from __future__ import annotations

import math


def _lg(v: float) -> float:
    return math.log2(v)


def mul_oaaconv(n: int, k: int) -> float:
    """Eq. (11): FFT, Hadamard product and inverse FFT multiplications of OaAConv."""
    f = 2 * k - 1
    return n * n / (k * k) * (2 * f * f * _lg(f * f) + f * f)


def add_oaaconv(n: int, k: int) -> float:
    """Eq. (12): FFT and inverse FFT additions plus the overlap additions."""
    f = 2 * k - 1
    return n * n / (k * k) * (2 * f * f * _lg(f * f) + k * k - k)


def mul_splitconv(n: int, k: int, s: int) -> float:
    """Eq. (13): multiplications of the split method with patch size s."""
    f = s + k - 1
    return n * n / (s * s) * (2 * f * f * _lg(f * f) + f * f)


def add_splitconv(n: int, k: int, s: int) -> float:
    """Eq. (14): additions of the split method (FFT and inverse FFT only)."""
    f = s + k - 1
    return n * n / (s * s) * (2 * f * f * _lg(f * f))
