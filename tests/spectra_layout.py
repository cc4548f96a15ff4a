"""Test-side helpers that re-index spectra between the oracle's full L x L
arrays and the library's stored-bin layout (documented in fftsplit.h).

Only index bookkeeping lives here -- no transform arithmetic: the stored
bins are a subset of the full spectrum (the four real bins of the columns
k2 = 0 and L/2 packed two to a slot, as real and imaginary part), and the
rest follows from the Hermitian symmetry of a real array's spectrum,
S[-k1, -k2] = conj(S[k1, k2]).
"""
import numpy as np


def stored_coords(L: int):
    """(k1, k2) of every complex stored bin, in the header's order; for even
    L the two slots that follow them hold the real bins of real_pairs(L).
    Odd L (the OaAConv sizes): columns k2 in [1, (L-1)/2], then k1 in
    [0, (L-1)/2] of column 0, nothing packed."""
    h2 = L // 2
    if L % 2:
        return [(k1, k2) for k2 in range(1, h2 + 1) for k1 in range(L)] + [(k1, 0) for k1 in range(h2 + 1)]
    out = [(k1, k2) for k2 in range(1, h2) for k1 in range(L)]
    out += [(k1, 0) for k1 in range(1, h2)]
    out += [(k1, h2) for k1 in range(1, h2)]
    return out


def real_pairs(L: int):
    """The last two stored slots: (bin in the real part, bin in the imaginary part)."""
    h2 = L // 2
    if L % 2:
        return []
    return [((0, 0), (h2, 0)), ((0, h2), (h2, h2))]


def full_to_stored(full: np.ndarray) -> np.ndarray:
    """[..., L, L] -> [bins, ...] (complex128)."""
    L = full.shape[-1]
    k1, k2 = np.array(stored_coords(L)).T
    st = np.moveaxis(full[..., k1, k2], -1, 0).astype(np.complex128)
    packed = [full[..., a[0], a[1]].real + 1j * full[..., b[0], b[1]].real for a, b in real_pairs(L)]
    return np.concatenate([st, np.stack(packed)], axis=0) if packed else st


def stored_to_full(stored: np.ndarray, L: int) -> np.ndarray:
    """[bins, ...] -> [..., L, L], filling the unstored bins by symmetry."""
    coords = stored_coords(L)
    nc = len(coords)
    lead = stored.shape[1:]
    full = np.zeros(lead + (L, L), dtype=np.complex128)
    have = np.zeros((L, L), dtype=bool)
    for f, (k1, k2) in enumerate(coords):
        full[..., k1, k2] = stored[f]
        have[k1, k2] = True
    for i, (a, b) in enumerate(real_pairs(L)):
        full[..., a[0], a[1]] = stored[nc + i].real
        full[..., b[0], b[1]] = stored[nc + i].imag
        have[a] = have[b] = True
    for k1 in range(L):
        for k2 in range(L):
            if not have[k1, k2]:
                m1, m2 = (-k1) % L, (-k2) % L
                assert have[m1, m2], (k1, k2)
                full[..., k1, k2] = np.conj(full[..., m1, m2])
    return full


def rel_l2(got, ref) -> float:
    """||got - ref|| / ||ref|| over all entries (complex entries by modulus)."""
    dt = np.complex128 if (np.iscomplexobj(got) or np.iscomplexobj(ref)) else np.float64
    got = np.asarray(got, dtype=dt)
    ref = np.asarray(ref, dtype=dt)
    den = np.linalg.norm(ref.ravel())
    return float(np.linalg.norm((got - ref).ravel()) / (den if den > 0 else 1.0))


def rel_max(got, ref) -> float:
    got = np.asarray(got)
    ref = np.asarray(ref)
    den = np.max(np.abs(ref)) if ref.size else 1.0
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0)) if ref.size else 0.0
