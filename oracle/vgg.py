"""VGG-16 convolution stack (test infrastructure only).

Section 4 runs the convolution layers of VGG16.  The stack here is the 13
3x3 'same' convolutions with bias and ReLU, and a 2x2 max-pool after
layers 2, 4, 7, 10 and 13.  Each layer is the direct cross-correlation of
eq. (1); float64 throughout.
"""
from __future__ import annotations

import numpy as np

from .direct import direct_xcorr2d
from .pool import maxpool2x2

POOL_AFTER = (2, 4, 7, 10, 13)


def vgg16_forward(x, layers, return_all=False):
    """Run the stack.  ``layers`` is a list of 13 (w, b) pairs.

    Returns the final activation, or with ``return_all`` the list of every
    layer's post-ReLU output (before pooling) followed by the final one.
    """
    a = np.asarray(x, dtype=np.float64)
    outs = []
    for i, (w, b) in enumerate(layers, start=1):
        a = direct_xcorr2d(a, w, b, relu=True)
        outs.append(a)
        if i in POOL_AFTER:
            a = maxpool2x2(a)
    return (outs, a) if return_all else a
