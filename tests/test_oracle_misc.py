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
