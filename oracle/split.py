"""FFT-based split convolution, step by step (test infrastructure only).

Follows Section 3.1 of the paper in its order:

1. Split the input into T x T patches d_i (eq. 4).  Tiles cover the image
   in a th x tw grid, th = ceil(H/T), tw = ceil(W/T); edge patches that run
   past the image see zeros (the paper is silent on ragged edges).
2. Pad each patch by p_i to an L x L patch, L = T + K - 1 (eqs. 5-6).  Two
   disciplines are implemented:
     * 'os'  (overlap-save, the paper's own flow): p_i is the P = K//2 wide
             border of neighbouring pixels, i.e. patches overlap by K//2 on
             each side; only pixels outside the image are zeros.
     * 'oaa' (overlap-add, Section 2 / Fig. 1, applied at tile size T):
             p_i is zeros, the T x T patch sits in the top-left corner.
3. Zero-pad the filter to L x L, top-left (eq. 8) and transform it.
4. Transform each patch and take the entry-wise (Hadamard) product with the
   filter spectrum (eq. 9).  Eq. (9) is single-channel; a layer with Cin
   inputs sums the Cin products per output channel, which is the same as
   summing the spatial results because the transform is linear.  CNN layers
   are cross-correlations, so the filter spectrum enters conjugated.
5. Inverse-transform, crop (eq. 10) and concatenate (the sentence after
   eq. 10) -- for 'os' the valid T x T corner of each patch is the output
   tile; for 'oaa' the whole L x L result is added into the output at the
   patch's offset, wrapped indices p >= T standing for p - L.

All arithmetic is float64/complex128 and uses the naive DFT of ``dft``.
"""
from __future__ import annotations

import math

import numpy as np

from .dft import dft2, idft2


def tile_grid(h: int, w: int, t: int):
    """Number of tile rows and columns covering an h x w image with T x T tiles."""
    if t <= 0:
        raise ValueError("tile size must be positive")
    return math.ceil(h / t), math.ceil(w / t)


def patch_windows(x, t: int, k: int, mode: str = "os") -> np.ndarray:
    """Steps 1-2: the padded patches, shape [n, th, tw, cin, L, L] (eqs. 4-6)."""
    x = np.asarray(x, dtype=np.float64)
    n, cin, h, wd = x.shape
    if k % 2 != 1:
        raise ValueError("odd kernel sizes only")
    p = k // 2
    L = t + k - 1
    th, tw = tile_grid(h, wd, t)
    # xbar: the image surrounded by enough zeros that every window slice is
    # in range (P before, the ragged tail plus P after).
    xbar = np.zeros((n, cin, th * t + 2 * p + L, tw * t + 2 * p + L))
    xbar[:, :, p:p + h, p:p + wd] = x
    out = np.zeros((n, th, tw, cin, L, L))
    for a in range(th):
        for b in range(tw):
            if mode == "os":
                # rows a*T - P .. a*T - P + L - 1 of the image; in xbar
                # coordinates that is a*T .. a*T + L - 1.
                out[:, a, b] = xbar[:, :, a * t:a * t + L, b * t:b * t + L]
            elif mode == "oaa":
                # rows a*T .. a*T + T - 1 of the image, then zeros.
                out[:, a, b, :, :t, :t] = xbar[:, :, a * t + p:a * t + p + t,
                                                b * t + p:b * t + p + t]
            else:
                raise ValueError(f"unknown mode {mode!r}")
    return out


def filter_spectra(w, L: int) -> np.ndarray:
    """Step 3: DFT of each K x K filter zero-padded top-left to L x L (eq. 8).

    Returns [cout, cin, L, L] complex (not conjugated).
    """
    w = np.asarray(w, dtype=np.float64)
    cout, cin, k, _ = w.shape
    if L < k:
        raise ValueError("FFT size smaller than the kernel")
    wpad = np.zeros((cout, cin, L, L))
    wpad[:, :, :k, :k] = w
    return dft2(wpad)


def patch_spectra(x, t: int, k: int, mode: str = "os") -> np.ndarray:
    """Steps 1-2 then the forward DFT of each patch: [n, th, tw, cin, L, L]."""
    return dft2(patch_windows(x, t, k, mode))


def hadamard_channel_sum(xs, ws) -> np.ndarray:
    """Step 4: Z[..., co, bins] = sum_ci Xs[..., ci, bins] * conj(Ws[co, ci, bins]) (eq. 9).

    xs: [..., cin, *bins] patch spectra (normally [n, th, tw, cin, L, L]);
    ws: [cout, cin, *bins] filter spectra with the same trailing bin axes.
    Returns [..., cout, *bins].
    """
    xs = np.asarray(xs, dtype=np.complex128)
    ws = np.asarray(ws, dtype=np.complex128)
    cout, cin = ws.shape[:2]
    bins = ws.shape[2:]
    lead = xs.shape[:xs.ndim - len(bins) - 1]
    if xs.shape[len(lead)] != cin or xs.shape[len(lead) + 1:] != bins:
        raise ValueError("patch and filter spectra do not match")
    nb = int(np.prod(bins)) if bins else 1
    npatch = int(np.prod(lead)) if lead else 1
    # For each frequency bin: the [patches x cin] matrix of patch spectra
    # times the [cin x cout] matrix of conjugated filter spectra.  Entry
    # (patch, co) is sum_ci Xs[patch, ci, bin] * conj(Ws[co, ci, bin]).
    xb = xs.reshape(npatch, cin, nb).transpose(2, 0, 1)          # [bins, P, cin]
    wb = np.conj(ws).reshape(cout, cin, nb).transpose(2, 1, 0)   # [bins, cin, cout]
    zb = np.matmul(xb, wb)                                       # [bins, P, cout]
    return np.ascontiguousarray(zb.transpose(1, 2, 0)).reshape(*lead, cout, *bins)


def inverse_place(z_spec, h: int, w: int, t: int, k: int, mode: str = "os",
                  b=None, relu: bool = False) -> np.ndarray:
    """Step 5: inverse DFT, crop / overlap-add, bias, ReLU (eq. 10).

    z_spec: [n, th, tw, cout, L, L].  Returns y [n, cout, h, w].
    """
    z = idft2(z_spec)
    scale = max(1.0, float(np.max(np.abs(z.real))) if z.size else 1.0)
    if z.size and float(np.max(np.abs(z.imag))) > 1e-9 * scale:
        raise AssertionError("inverse of a real layer's spectrum is not real")
    z = z.real
    n, th, tw, cout, L, _ = z.shape
    p = k // 2
    # Output canvas with room for ragged tiles and overlap-add spill on both
    # sides; the image occupies rows/cols [L, L + h).
    off = L
    canvas = np.zeros((n, cout, th * t + 2 * L, tw * t + 2 * L))
    for a in range(th):
        for bb in range(tw):
            if mode == "os":
                # crop: the first T x T entries are the valid outputs of the
                # tile whose top-left output pixel is (a*T, b*T).
                r0, c0 = off + a * t, off + bb * t
                canvas[:, :, r0:r0 + t, c0:c0 + t] = z[:, a, bb, :, :t, :t]
            elif mode == "oaa":
                # entry (p, q) adds into output (a*T + P + p', b*T + P + q')
                # with p' = p for p < T and p' = p - L for p >= T.
                for pi in range(L):
                    pr = pi if pi < t else pi - L
                    r = off + a * t + p + pr
                    for qi in range(L):
                        qr = qi if qi < t else qi - L
                        c = off + bb * t + p + qr
                        canvas[:, :, r, c] += z[:, a, bb, :, pi, qi]
            else:
                raise ValueError(f"unknown mode {mode!r}")
    y = canvas[:, :, off:off + h, off:off + w].copy()
    if b is not None:
        y = y + np.asarray(b, dtype=np.float64)[None, :, None, None]
    if relu:
        y = np.maximum(y, 0.0)
    return y


def split_conv(x, w, b=None, t: int = 6, mode: str = "os", relu: bool = False) -> np.ndarray:
    """The whole method of Section 3.1 for one layer: y [n, cout, h, w], float64."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, cin, h, wd = x.shape
    cout, cin_w, k, k2 = w.shape
    if cin != cin_w or k != k2:
        raise ValueError("shape mismatch")
    L = t + k - 1
    xs = patch_spectra(x, t, k, mode)
    ws = filter_spectra(w, L)
    zs = hadamard_channel_sum(xs, ws)
    return inverse_place(zs, h, wd, t, k, mode, b, relu)
