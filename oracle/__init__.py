"""CPU oracle for the FFT-based split convolution (arXiv:2003.12621).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 NumPy
implementation of what the GPU path computes.  Only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it; the product
library never calls it and shares no code, tables or constants with it.

Contents (each function cites the passage of the paper it follows):

* ``direct``  -- the direct spatial cross-correlation of Section 2, eq. (1),
  which defines the result the split method must reproduce; plus a scalar
  seven-loop brute force for tiny inputs.
* ``dft``     -- the 2-D DFT of eq. (3) written out as a matrix product.
* ``split``   -- the splitting method of Section 3.1, eqs. (4)-(10): split,
  pad, transform, Hadamard product (summed over input channels), inverse
  transform, crop and concatenate; and the overlap-add discipline of
  Section 2 / Fig. 1 applied at tile size T.
* ``pool``    -- 2x2 stride-2 max-pooling between VGG stages.
* ``vgg``     -- the 13-layer VGG-16 convolution stack built from the above.
* ``opcount`` -- the operation-count closed forms of Section 3.2,
  eqs. (11)-(14).

Every function here is pinned by the CPU tests against something other than
itself: brute force, closed forms, invariants or a library routine.
"""
from .direct import direct_xcorr2d, brute_xcorr2d
from .dft import dft_matrix, dft2, idft2
from .split import (
    tile_grid,
    patch_windows,
    filter_spectra,
    patch_spectra,
    hadamard_channel_sum,
    inverse_place,
    split_conv,
)
from .pool import maxpool2x2
from .vgg import vgg16_forward
from . import opcount

__all__ = [
    "direct_xcorr2d",
    "brute_xcorr2d",
    "dft_matrix",
    "dft2",
    "idft2",
    "tile_grid",
    "patch_windows",
    "filter_spectra",
    "patch_spectra",
    "hadamard_channel_sum",
    "inverse_place",
    "split_conv",
    "maxpool2x2",
    "vgg16_forward",
    "opcount",
]
