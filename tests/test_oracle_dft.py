"""Pins for the oracle's naive 2-D DFT (eq. 3, unnormalised forward, 1/L^2 inverse)."""
import numpy as np
import pytest

import oracle

LS = [1, 2, 3, 5, 8, 16, 32]


@pytest.mark.parametrize("L", LS)
def test_delta_transforms_to_ones(L):
    a = np.zeros((L, L))
    a[0, 0] = 1.0
    np.testing.assert_allclose(oracle.dft2(a), np.ones((L, L)), rtol=0, atol=1e-13)


@pytest.mark.parametrize("L", LS)
def test_matches_numpy_fft2(L):
    rng = np.random.default_rng(L)
    a = rng.standard_normal((3, L, L)) + 1j * rng.standard_normal((3, L, L))
    np.testing.assert_allclose(oracle.dft2(a), np.fft.fft2(a), rtol=0, atol=1e-11 * L * L)
    np.testing.assert_allclose(oracle.idft2(a), np.fft.ifft2(a), rtol=0, atol=1e-12)


@pytest.mark.parametrize("L", [8, 16, 32])
def test_complex_exponential_is_one_spike(L):
    # a[m, n] = exp(+2 pi i (m k0 + n l0) / L) has all of its energy in bin (k0, l0).
    k0, l0 = 3, L - 2
    m = np.arange(L)
    a = np.exp(2j * np.pi * (np.outer(m, np.ones(L)) * k0 + np.outer(np.ones(L), m) * l0) / L)
    spec = oracle.dft2(a)
    expect = np.zeros((L, L), dtype=complex)
    expect[k0, l0] = L * L
    np.testing.assert_allclose(spec, expect, rtol=0, atol=1e-10)


@pytest.mark.parametrize("L", [4, 8, 16, 32])
def test_linearity_parseval_roundtrip_hermitian(L):
    rng = np.random.default_rng(100 + L)
    a = rng.standard_normal((L, L))
    b = rng.standard_normal((L, L))
    A, B = oracle.dft2(a), oracle.dft2(b)
    np.testing.assert_allclose(oracle.dft2(2.0 * a - 3.0 * b), 2.0 * A - 3.0 * B, rtol=0, atol=1e-11)
    # Parseval: sum |a|^2 = sum |A|^2 / L^2
    assert abs(np.sum(a * a) - np.sum(np.abs(A) ** 2) / (L * L)) < 1e-10 * np.sum(a * a)
    np.testing.assert_allclose(oracle.idft2(A).real, a, rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle.idft2(A).imag, 0.0, rtol=0, atol=1e-12)
    # Hermitian symmetry of a real input's spectrum: A[-k, -l] = conj(A[k, l])
    neg = (-np.arange(L)) % L
    np.testing.assert_allclose(A[np.ix_(neg, neg)], np.conj(A), rtol=0, atol=1e-11)


def test_circular_convolution_theorem():
    # The product of two spectra is the spectrum of the circular convolution.
    L = 8
    rng = np.random.default_rng(9)
    a = rng.standard_normal((L, L))
    b = rng.standard_normal((L, L))
    conv = np.zeros((L, L))
    for i in range(L):
        for j in range(L):
            for m in range(L):
                for n in range(L):
                    conv[i, j] += a[m, n] * b[(i - m) % L, (j - n) % L]
    got = oracle.idft2(oracle.dft2(a) * oracle.dft2(b)).real
    np.testing.assert_allclose(got, conv, rtol=0, atol=1e-11)


def test_rejects_non_square():
    with pytest.raises(ValueError):
        oracle.dft2(np.zeros((4, 5)))
