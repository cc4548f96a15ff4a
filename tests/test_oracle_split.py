"""Pins for the oracle's split method (Section 3.1, eqs. 4-10).

The split result must equal the direct cross-correlation for every tile
size, in both the overlap-save (crop and concatenate) and the overlap-add
disciplines; each stage is also checked against a brute-force loop or a
library routine so that a failure localises.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from workloads import small_layer, make_config, CONFIGS


TINY = [
    # n, cin, h, w, cout, k
    (1, 1, 5, 5, 1, 1),
    (1, 2, 7, 5, 3, 3),
    (2, 3, 6, 9, 2, 3),
    (1, 2, 8, 7, 2, 5),
    (1, 1, 4, 4, 2, 5),
]


@pytest.mark.parametrize("shape", TINY)
@pytest.mark.parametrize("mode", ["os", "oaa"])
def test_split_equals_direct_for_every_tile_size(shape, mode):
    n, cin, h, w, cout, k = shape
    x, wt = small_layer(n, cin, h, w, cout, k, seed=11)
    b = np.linspace(-0.2, 0.3, cout)
    ref = oracle.direct_xcorr2d(x, wt, b)
    scale = np.max(np.abs(ref))
    for t in range(1, max(h, w) + 3):
        got = oracle.split_conv(x, wt, b, t=t, mode=mode)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * scale, err_msg=f"T={t}")


@pytest.mark.parametrize("t", [6, 7, 14, 30, 32])
def test_overlap_save_equals_overlap_add(t):
    x, wt = small_layer(1, 3, 32, 29, 4, 3, seed=12)
    os_ = oracle.split_conv(x, wt, t=t, mode="os")
    oaa = oracle.split_conv(x, wt, t=t, mode="oaa")
    np.testing.assert_allclose(os_, oaa, rtol=0, atol=1e-12 * np.max(np.abs(os_)))


def test_first_config_tile_invariance_and_relu():
    # The 1x3x32x32 -> 16 layer: 36 patches per channel at T = 6 (L = 8),
    # and every other tile size gives the same result.
    x, w, b = make_config("c1_32x3")
    assert oracle.tile_grid(32, 32, 6) == (6, 6)
    ref = oracle.direct_xcorr2d(x, w, b, relu=True)
    for t in (1, 2, 6, 14, 30, 32, 33):
        for mode in ("os", "oaa"):
            got = oracle.split_conv(x, w, b, t=t, mode=mode, relu=True)
            np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * np.max(np.abs(ref)))


def test_single_tile_is_whole_image_fft_convolution():
    # T >= H, W: one patch covers the image -- the conventional FFT
    # convolution of eq. (2) on the zero-padded image.
    x, wt = small_layer(1, 2, 9, 9, 2, 3, seed=13)
    ref = oracle.direct_xcorr2d(x, wt)
    th, tw = oracle.tile_grid(9, 9, 9)
    assert (th, tw) == (1, 1)
    got = oracle.split_conv(x, wt, t=9, mode="os")
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * np.max(np.abs(ref)))


@pytest.mark.parametrize("mode", ["os", "oaa"])
def test_patch_windows_brute_force(mode):
    x, _ = small_layer(2, 2, 7, 10, 1, 3, seed=14)
    for k, t in [(3, 3), (5, 4), (3, 6), (1, 5)]:
        p = k // 2
        L = t + k - 1
        win = oracle.patch_windows(x, t, k, mode)
        th, tw = oracle.tile_grid(7, 10, t)
        assert win.shape == (2, th, tw, 2, L, L)
        for a in range(th):
            for b in range(tw):
                for m in range(L):
                    for q in range(L):
                        if mode == "os":
                            r, c = a * t - p + m, b * t - p + q
                            inside = 0 <= r < 7 and 0 <= c < 10
                        else:
                            r, c = a * t + m, b * t + q
                            inside = m < t and q < t and r < 7 and c < 10
                        expect = x[:, :, r, c] if inside else 0.0
                        np.testing.assert_array_equal(win[:, a, b, :, m, q], expect)


@pytest.mark.parametrize("L,k", [(8, 3), (16, 5), (32, 3), (5, 5)])
def test_filter_spectra_matches_numpy_fft(L, k):
    rng = np.random.default_rng(15)
    w = rng.standard_normal((3, 2, k, k))
    pad = np.zeros((3, 2, L, L))
    pad[:, :, :k, :k] = w
    np.testing.assert_allclose(oracle.filter_spectra(w, L), np.fft.fft2(pad), rtol=0, atol=1e-11)


def test_hadamard_channel_sum_brute_force():
    rng = np.random.default_rng(16)
    xs = rng.standard_normal((2, 2, 3, 4, 5, 5)) + 1j * rng.standard_normal((2, 2, 3, 4, 5, 5))
    ws = rng.standard_normal((3, 4, 5, 5)) + 1j * rng.standard_normal((3, 4, 5, 5))
    got = oracle.hadamard_channel_sum(xs, ws)
    assert got.shape == (2, 2, 3, 3, 5, 5)
    for n in range(2):
        for a in range(2):
            for b in range(3):
                for co in range(3):
                    acc = np.zeros((5, 5), dtype=complex)
                    for ci in range(4):
                        acc += xs[n, a, b, ci] * np.conj(ws[co, ci])
                    np.testing.assert_allclose(got[n, a, b, co], acc, rtol=0, atol=1e-12)


@pytest.mark.parametrize("mode", ["os", "oaa"])
def test_inverse_place_brute_force(mode):
    # Known spatial tiles z go through the (pinned) forward DFT; placing the
    # inverse must put entry (p, q) of tile (a, b) where the text says.
    rng = np.random.default_rng(17)
    n, cout, h, w, t, k = 1, 2, 9, 8, 4, 3
    L, p = t + k - 1, k // 2
    th, tw = oracle.tile_grid(h, w, t)
    z = rng.standard_normal((n, th, tw, cout, L, L))
    got = oracle.inverse_place(oracle.dft2(z), h, w, t, k, mode)
    expect = np.zeros((n, cout, h, w))
    for a in range(th):
        for b in range(tw):
            for pi in range(L):
                for qi in range(L):
                    if mode == "os":
                        if pi >= t or qi >= t:
                            continue
                        r, c = a * t + pi, b * t + qi
                        if r < h and c < w:
                            expect[:, :, r, c] = z[:, a, b, :, pi, qi]
                    else:
                        pr = pi if pi < t else pi - L
                        qr = qi if qi < t else qi - L
                        r, c = a * t + p + pr, b * t + p + qr
                        if 0 <= r < h and 0 <= c < w:
                            expect[:, :, r, c] += z[:, a, b, :, pi, qi]
    np.testing.assert_allclose(got, expect, rtol=0, atol=1e-12)


@settings(max_examples=40, deadline=None)
@given(
    n=st.integers(1, 2), cin=st.integers(1, 3), cout=st.integers(1, 3),
    h=st.integers(1, 11), w=st.integers(1, 11), k=st.sampled_from([1, 3, 5]),
    t=st.integers(1, 13), mode=st.sampled_from(["os", "oaa"]), seed=st.integers(0, 2**31 - 1),
)
def test_property_split_equals_direct(n, cin, cout, h, w, k, t, mode, seed):
    x, wt = small_layer(n, cin, h, w, cout, k, seed=seed)
    ref = oracle.direct_xcorr2d(x, wt)
    got = oracle.split_conv(x, wt, t=t, mode=mode)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * max(1.0, np.max(np.abs(ref))))


@pytest.mark.slow
def test_mid_size_layer_tile_sizes_agree():
    # A 224^2 x 8 -> 8 slice of the 224^2 x 64 layer, at every tile size used
    # for it (FFT sizes 8, 16, 32), against direct correlation.
    x, w, _ = make_config("c2_224x64")
    x, w = x[:, :8], w[:8, :8]
    ref = oracle.direct_xcorr2d(x, w)
    for t in CONFIGS["c2_224x64"]["tiles"]:
        got = oracle.split_conv(x, w, t=t, mode="os")
        err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        assert err < 1e-13, (t, err)
