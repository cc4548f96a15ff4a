"""Naive 2-D discrete Fourier transform (test infrastructure only).

Section 2, eq. (3) defines the 2-D transform of an L x L array.  As printed,
its exponent carries 2*pi*i/N^2 and its forward sum a 1/N^2 factor; neither
gives a transform whose Hadamard product is a convolution.  The reading used
here is the standard one: an unnormalised forward transform

    A[k, l] = sum_{m, n < L} a[m, n] * exp(-2*pi*i*(m*k + n*l) / L)

and an inverse that carries the single 1/L^2 factor.

It is computed as D @ a @ D^T with D[k, m] = exp(-2*pi*i*((k*m) mod L)/L):
no FFT, no reordering.  The product k*m is reduced mod L before the
exponential so that large arguments do not lose accuracy.  float64/complex128.
"""
from __future__ import annotations

import numpy as np


def dft_matrix(L: int) -> np.ndarray:
    """D[k, m] = exp(-2*pi*i*((k*m) mod L)/L), complex128, L x L."""
    k = np.arange(L)
    km = np.outer(k, k) % L
    return np.exp(-2j * np.pi * km / L)


def dft2(a) -> np.ndarray:
    """Unnormalised forward 2-D DFT over the last two (square) axes."""
    a = np.asarray(a)
    L = a.shape[-1]
    if a.shape[-2] != L:
        raise ValueError("dft2 expects square trailing axes")
    d = dft_matrix(L)
    return d @ a.astype(np.complex128) @ d.T


def idft2(spec) -> np.ndarray:
    """Inverse 2-D DFT over the last two axes, with the 1/L^2 factor."""
    spec = np.asarray(spec, dtype=np.complex128)
    L = spec.shape[-1]
    if spec.shape[-2] != L:
        raise ValueError("idft2 expects square trailing axes")
    dc = np.conj(dft_matrix(L))
    return dc @ spec @ dc.T / float(L * L)
