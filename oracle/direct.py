"""Direct spatial cross-correlation (test infrastructure only).

Section 2, eq. (1) writes the layer as y = d (x) w.  In a CNN the operator is
a cross-correlation with OIHW weights, and a 'same' layer pads the input with
K//2 zeros on every side, so for odd K, P = K//2:

    y[n, co, i, j] = b[co] + sum_ci sum_{u,v < K} w[co, ci, u, v] * xbar[n, ci, i+u-P, j+v-P]

where xbar equals x inside the image and 0 outside.  This is the result the
split method reproduces (up to rounding), so it is the oracle's definition of
the layer.  All arithmetic is float64.
"""
from __future__ import annotations

import numpy as np


def _check(x, w):
    if x.ndim != 4 or w.ndim != 4:
        raise ValueError("x must be [n, cin, h, w] and w [cout, cin, k, k]")
    n, cin, h, wd = x.shape
    cout, cin_w, k, k2 = w.shape
    if cin != cin_w or k != k2 or k % 2 != 1:
        raise ValueError("channel mismatch, non-square or even kernel")
    return n, cin, h, wd, cout, k


def direct_xcorr2d(x, w, b=None, relu=False):
    """Eq. (1) as 'same' cross-correlation, float64.

    The K*K taps are summed one shifted view at a time; each tap is a
    contraction over input channels done by ``numpy.tensordot``.
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, cin, h, wd, cout, k = _check(x, w)
    p = k // 2
    xbar = np.zeros((n, cin, h + 2 * p, wd + 2 * p))
    xbar[:, :, p:p + h, p:p + wd] = x
    y = np.zeros((cout, n, h, wd))
    for u in range(k):
        for v in range(k):
            view = xbar[:, :, u:u + h, v:v + wd]          # xbar[i+u-P, j+v-P]
            y += np.tensordot(w[:, :, u, v], view, axes=([1], [1]))
    y = y.transpose(1, 0, 2, 3)
    if b is not None:
        y = y + np.asarray(b, dtype=np.float64)[None, :, None, None]
    if relu:
        y = np.maximum(y, 0.0)
    return np.ascontiguousarray(y)


def brute_xcorr2d(x, w, b=None, relu=False):
    """The same sum as ``direct_xcorr2d``, one scalar term at a time.

    Seven nested Python loops: only for tiny inputs.  Out-of-image taps are
    skipped, which is the zero padding.
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, cin, h, wd, cout, k = _check(x, w)
    p = k // 2
    y = np.zeros((n, cout, h, wd))
    for img in range(n):
        for co in range(cout):
            for i in range(h):
                for j in range(wd):
                    acc = 0.0 if b is None else float(b[co])
                    for ci in range(cin):
                        for u in range(k):
                            for v in range(k):
                                r, c = i + u - p, j + v - p
                                if 0 <= r < h and 0 <= c < wd:
                                    acc += w[co, ci, u, v] * x[img, ci, r, c]
                    y[img, co, i, j] = max(acc, 0.0) if relu else acc
    return y
