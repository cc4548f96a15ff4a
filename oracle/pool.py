"""2x2, stride-2 max-pooling (test infrastructure only).

Not part of the split method: VGG-16 places one such pool after each of its
five convolution stages, which the paper's VGG16 experiment (Section 4)
runs through.  Odd trailing rows/columns are dropped (floor).
"""
from __future__ import annotations

import numpy as np


def maxpool2x2(x) -> np.ndarray:
    x = np.asarray(x)
    n, c, h, w = x.shape
    ho, wo = h // 2, w // 2
    v = x[:, :, :2 * ho, :2 * wo].reshape(n, c, ho, 2, wo, 2)
    return v.max(axis=(3, 5))
