"""Pins for the oracle's direct cross-correlation (eq. 1 read as a CNN layer).

Each check comes from outside the function under test: a scalar brute force,
PyTorch's own conv2d (a library special case), closed forms and linearity.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import small_layer

SHAPES = [
    # n, cin, h, w, cout, k
    (1, 1, 5, 5, 1, 1),
    (1, 1, 5, 7, 1, 3),
    (2, 2, 6, 4, 3, 3),
    (1, 3, 7, 6, 2, 5),
    (2, 1, 3, 3, 2, 5),   # kernel wider than the image
]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("relu", [False, True])
def test_direct_matches_brute_force(shape, relu):
    n, cin, h, w, cout, k = shape
    x, wt = small_layer(n, cin, h, w, cout, k, seed=1)
    b = np.linspace(-0.5, 0.5, cout).astype(np.float32)
    got = oracle.direct_xcorr2d(x, wt, b, relu=relu)
    ref = oracle.brute_xcorr2d(x, wt, b, relu=relu)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES + [(2, 8, 17, 13, 5, 3), (1, 4, 12, 12, 6, 7)])
def test_direct_matches_torch_conv2d(shape):
    n, cin, h, w, cout, k = shape
    x, wt = small_layer(n, cin, h, w, cout, k, seed=2)
    b = np.arange(cout, dtype=np.float32) * 0.25 - 0.3
    got = oracle.direct_xcorr2d(x, wt, b)
    ref = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(wt).double(),
                                     torch.from_numpy(b).double(), stride=1, padding=k // 2).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k", [1, 3, 5])
def test_centred_delta_kernel_is_identity(k):
    x, _ = small_layer(2, 3, 9, 7, 3, k, seed=3)
    w = np.zeros((3, 3, k, k))
    for c in range(3):
        w[c, c, k // 2, k // 2] = 1.0
    np.testing.assert_array_equal(oracle.direct_xcorr2d(x, w), x.astype(np.float64))


@pytest.mark.parametrize("k", [3, 5])
def test_delta_input_gives_flipped_kernel(k):
    # A unit impulse at (i0, j0) makes y[i0 + P - u, j0 + P - v] = w[u, v]:
    # the kernel rotated by 180 degrees around the impulse.
    h = w_ = 11
    i0, j0 = 5, 4
    x = np.zeros((1, 1, h, w_))
    x[0, 0, i0, j0] = 1.0
    rng = np.random.default_rng(4)
    wt = rng.standard_normal((1, 1, k, k))
    y = oracle.direct_xcorr2d(x, wt)[0, 0]
    p = k // 2
    expect = np.zeros((h, w_))
    for u in range(k):
        for v in range(k):
            expect[i0 + p - u, j0 + p - v] = wt[0, 0, u, v]
    np.testing.assert_allclose(y, expect, rtol=0, atol=1e-15)


@pytest.mark.parametrize("k", [3, 5])
def test_all_ones_counts_in_image_taps(k):
    cin, h, w_ = 3, 8, 10
    y = oracle.direct_xcorr2d(np.ones((1, cin, h, w_)), np.ones((2, cin, k, k)))
    p = k // 2
    for i in range(h):
        for j in range(w_):
            rows = min(i + p, h - 1) - max(i - p, 0) + 1
            cols = min(j + p, w_ - 1) - max(j - p, 0) + 1
            assert y[0, 0, i, j] == cin * rows * cols
            assert y[0, 1, i, j] == cin * rows * cols
    assert y[0, 0, h // 2, w_ // 2] == cin * k * k


def test_linearity():
    x1, w1 = (v.astype(np.float64) for v in small_layer(1, 2, 8, 9, 3, 3, seed=5))
    x2, w2 = (v.astype(np.float64) for v in small_layer(1, 2, 8, 9, 3, 3, seed=6))
    a, c = 0.7, -1.3
    lhs = oracle.direct_xcorr2d(a * x1 + c * x2, w1)
    rhs = a * oracle.direct_xcorr2d(x1, w1) + c * oracle.direct_xcorr2d(x2, w1)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12, atol=1e-12)
    lhs = oracle.direct_xcorr2d(x1, a * w1 + c * w2)
    rhs = a * oracle.direct_xcorr2d(x1, w1) + c * oracle.direct_xcorr2d(x1, w2)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12, atol=1e-12)


def test_bias_and_relu():
    x, w = small_layer(1, 2, 6, 6, 2, 3, seed=7)
    b = np.array([0.5, -0.25])
    base = oracle.direct_xcorr2d(x, w)
    np.testing.assert_allclose(oracle.direct_xcorr2d(x, w, b), base + b[None, :, None, None], rtol=0, atol=1e-15)
    np.testing.assert_array_equal(oracle.direct_xcorr2d(x, w, b, relu=True),
                                  np.maximum(base + b[None, :, None, None], 0.0))


def test_rejects_even_kernel():
    with pytest.raises(ValueError):
        oracle.direct_xcorr2d(np.zeros((1, 1, 4, 4)), np.zeros((1, 1, 2, 2)))
