"""Test-side helpers that re-index spectra between the oracle's full L x L
arrays and the library's stored-bin layout (documented in fftsplit.h).

Only index bookkeeping lives here -- no transform arithmetic: the stored
bins are a subset of the full spectrum, and the rest follows from the
Hermitian symmetry of a real array's spectrum, S[-k1, -k2] = conj(S[k1, k2]).
"""
import numpy as np


def stored_coords(L: int):
    """(k1, k2) of every stored bin in the header's order."""
    h2 = L // 2
    out = [(k1, k2) for k2 in range(1, h2) for k1 in range(L)]
    out += [(k1, 0) for k1 in range(h2 + 1)]
    out += [(k1, h2) for k1 in range(h2 + 1)]
    return out


def full_to_stored(full: np.ndarray) -> np.ndarray:
    """[..., L, L] -> [bins, ...]."""
    L = full.shape[-1]
    k1, k2 = np.array(stored_coords(L)).T
    return np.moveaxis(full[..., k1, k2], -1, 0)


def stored_to_full(stored: np.ndarray, L: int) -> np.ndarray:
    """[bins, ...] -> [..., L, L], filling the unstored bins by symmetry."""
    coords = stored_coords(L)
    lead = stored.shape[1:]
    full = np.zeros(lead + (L, L), dtype=np.complex128)
    have = np.zeros((L, L), dtype=bool)
    for f, (k1, k2) in enumerate(coords):
        full[..., k1, k2] = stored[f]
        have[k1, k2] = True
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
