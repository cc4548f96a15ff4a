"""Pins for the oracle's max-pool, VGG stack and operation counts."""
import numpy as np
import pytest
import torch

import oracle
from oracle import opcount


def test_maxpool_matches_torch():
    rng = np.random.default_rng(21)
    for shape in [(2, 3, 8, 8), (1, 2, 7, 9), (1, 1, 2, 2), (1, 1, 3, 2)]:
        x = rng.standard_normal(shape)
        ref = torch.nn.functional.max_pool2d(torch.from_numpy(x), 2, 2).numpy()
        np.testing.assert_array_equal(oracle.maxpool2x2(x), ref)


def test_vgg_stack_matches_torch_on_a_thin_net():
    rng = np.random.default_rng(22)
    chans = [(2, 3), (3, 3), (3, 4), (4, 4), (4, 5), (5, 5), (5, 5),
             (5, 6), (6, 6), (6, 6), (6, 4), (4, 4), (4, 3)]
    layers = [(rng.standard_normal((co, ci, 3, 3)) * 0.4, rng.uniform(-0.1, 0.1, co)) for ci, co in chans]
    x = rng.uniform(0, 1, (2, 2, 32, 32))
    got = oracle.vgg16_forward(x, layers)
    t = torch.from_numpy(x)
    for i, (w, b) in enumerate(layers, start=1):
        t = torch.relu(torch.nn.functional.conv2d(t, torch.from_numpy(w), torch.from_numpy(b), padding=1))
        if i in (2, 4, 7, 10, 13):
            t = torch.nn.functional.max_pool2d(t, 2, 2)
    assert got.shape == (2, 3, 1, 1)
    np.testing.assert_allclose(got, t.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("n,k", [(56, 3), (56, 5), (224, 3), (224, 5), (32, 7)])
def test_opcount_split_with_kernel_sized_patches_matches_oaaconv(n, k):
    # Section 3.2: with the patch size equal to the kernel size the split
    # method has the OaAConv multiplication count; its additions lack only
    # the overlap additions (the k^2 - k term of eq. 12).
    assert opcount.mul_splitconv(n, k, k) == pytest.approx(opcount.mul_oaaconv(n, k), rel=1e-15)
    diff = opcount.add_oaaconv(n, k) - opcount.add_splitconv(n, k, k)
    assert diff == pytest.approx(n * n / (k * k) * (k * k - k), rel=1e-12)


@pytest.mark.parametrize("n", [56, 112, 224])
def test_opcount_split_below_oaaconv_and_gap_grows_with_kernel(n):
    # Fig. 3's stated outcome: for S = 16 and 32 the split method needs fewer
    # operations than OaAConv, and the gap widens as the kernel grows over
    # the usual CNN kernel sizes 3, 5, 7.  (For S = 16 the formulas make the
    # gap shrink again beyond k = 7; the figure's kernel range is not given.)
    for s in (16, 32):
        gaps = []
        for k in (3, 5, 7, 9, 11):
            split = opcount.mul_splitconv(n, k, s) + opcount.add_splitconv(n, k, s)
            oaa = opcount.mul_oaaconv(n, k) + opcount.add_oaaconv(n, k)
            gaps.append(oaa - split)
        assert all(g > 0 for g in gaps)
        assert gaps[0] < gaps[1] < gaps[2]


# Values derived by hand from Section 3.2's definitions, at points where the
# squared transform size is a power of two, so its base-2 logarithm (the
# number of radix-2 stages of a 2-D transform of f*f points) is an integer.
# Per (input, output) channel pair, an N x N image holds N^2/s^2 patches;
# each costs a forward and an inverse transform of f*f points, f = s + k - 1,
# with f*f operations per radix-2 stage and log2(f*f) stages (the
# 2 f^2 log f^2 term), and for the multiplications one Hadamard product per
# point (the f^2 term).  Eq. (14) has no Hadamard or overlap term.
#
#   N = 24, k = 3, s = 6:  f = 8,  f^2 = 64,   log2 = 6,  16 patches
#       MUL = 16 * (2*64*6 + 64)      = 16 * 832    = 13312
#       ADD = 16 * (2*64*6)           = 16 * 768    = 12288
#   N = 32, k = 1, s = 16: f = 16, f^2 = 256,  log2 = 8,  4 patches
#       MUL = 4 * (2*256*8 + 256)     = 4 * 4352    = 17408
#       ADD = 4 * 4096                              = 16384
#   N = 56, k = 5, s = 28: f = 32, f^2 = 1024, log2 = 10, 4 patches
#       MUL = 4 * (2*1024*10 + 1024)  = 4 * 21504   = 86016
#       ADD = 4 * 20480                             = 81920
#   N = 64, k = 3, s = 30: f = 32, 64^2/30^2 = 4096/900 patches (eq. 13 does
#       not round the patch count)
#       MUL = 4096/900 * 21504 = 88080384/900,  ADD = 4096/900 * 20480
SPLIT_BY_HAND = [
    # (N, k, s, MUL, ADD)
    (24, 3, 6, 13312.0, 12288.0),
    (32, 1, 16, 17408.0, 16384.0),
    (56, 5, 28, 86016.0, 81920.0),
    (64, 3, 30, 88080384.0 / 900.0, 4096.0 * 20480.0 / 900.0),
]


@pytest.mark.parametrize("n,k,s,mul,add", SPLIT_BY_HAND)
def test_opcount_split_values_derived_by_hand(n, k, s, mul, add):
    assert opcount.mul_splitconv(n, k, s) == pytest.approx(mul, rel=1e-14)
    assert opcount.add_splitconv(n, k, s) == pytest.approx(add, rel=1e-14)


def test_opcount_oaaconv_values_derived_by_hand():
    # Eqs. (11)-(12) with k = 1: f = 2k - 1 = 1, a one-point transform has
    # log2(1) = 0 stages, so only the N^2 Hadamard products remain, and the
    # k^2 - k overlap additions vanish (a 1 x 1 kernel's patches do not
    # overlap).
    assert opcount.mul_oaaconv(10, 1) == 100.0
    assert opcount.add_oaaconv(10, 1) == 0.0
    # k = 3 (f = 5): log2(25) = 2 log2(5) = 4.643856189774724; N = 6 holds
    # 36/9 = 4 patches, each with 2*25*4.643856189774724 = 232.1928094887362
    # transform operations, plus 25 Hadamard products (eq. 11) or
    # 9 - 3 = 6 overlap additions (eq. 12).
    assert opcount.mul_oaaconv(6, 3) == pytest.approx(4 * (232.1928094887362 + 25), rel=1e-14)
    assert opcount.add_oaaconv(6, 3) == pytest.approx(4 * (232.1928094887362 + 6), rel=1e-14)
    # The overlap additions alone: 4 patches x (k^2 - k) = 24.
    assert opcount.add_oaaconv(6, 3) - opcount.add_splitconv(6, 3, 3) == pytest.approx(24.0, rel=1e-12)


def test_opcount_golden_table():
    # tests/golden/opcounts.txt is written by tests/golden/make_golden.py,
    # which calls only oracle.opcount.
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "opcounts.txt")
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    assert rows
    for name, n, k, s, val in rows:
        n, k, s, val = int(n), int(k), int(s), float(val)
        fn = getattr(opcount, name)
        got = fn(n, k) if s == 0 else fn(n, k, s)
        assert got == pytest.approx(val, rel=1e-9), (name, n, k, s)
