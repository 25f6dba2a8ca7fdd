"""TEST INFRASTRUCTURE ONLY -- oracle of the multi-mode SVD invariants (Section
4.2, "Matching Equivalent Tensors").

For an r-way tensor T and a non-empty proper subset G of its modes, the
unfolding T_(G) has the modes in G (in increasing order) as rows and the
others (in increasing order) as columns; its singular values, in descending
order, are sigma(T_(G)).  The invariant set collects sigma(T_(G)) over every
such G.  Transposing an unfolding does not change its singular values and
T_(G^c) is the transpose of T_(G), so the set is carried by the subsets that
contain mode 0 (2^(r-1) - 1 of them); this oracle lists those, in increasing
order of the bit mask of G.  Singular values come from numpy's SVD in fp64
(the data widened exactly from fp32).

Two tensors match when their invariant sets match: their lists can be paired
one to one so that paired spectra have the same length and differ by at most
eps x (the larger leading singular value of the two) in every position.  The
pairing is searched exhaustively (augmenting paths over at most 15 x 15
candidates).
"""
from __future__ import annotations

import numpy as np


def canonical_masks(rank: int) -> list:
    """Bit masks of the non-empty proper mode subsets that contain mode 0."""
    return [g for g in range(1, (1 << rank) - 1) if g & 1]


def unfold(T: np.ndarray, mask: int) -> np.ndarray:
    """T_(G): modes of G as rows, the others as columns (both in increasing order)."""
    r = T.ndim
    rows = [i for i in range(r) if mask >> i & 1]
    cols = [i for i in range(r) if not mask >> i & 1]
    M = int(np.prod([T.shape[i] for i in rows]))
    N = int(np.prod([T.shape[i] for i in cols]))
    return np.transpose(T, rows + cols).reshape(M, N)


def invariants(T) -> list:
    """The spectra sigma(T_(G)) of the canonical unfoldings, each descending."""
    T = np.asarray(T, dtype=np.float64)
    return [np.linalg.svd(unfold(T, g), compute_uv=False) for g in canonical_masks(T.ndim)]


def spectra_close(a: np.ndarray, b: np.ndarray, eps: float) -> bool:
    if a.shape != b.shape:
        return False
    if a.size == 0:
        return True
    scale = max(float(a[0]), float(b[0]))
    return bool(np.all(np.abs(a - b) <= eps * scale))


def match(sa: list, sb: list, eps: float) -> bool:
    """One-to-one pairing of two invariant lists with every pair close."""
    if len(sa) != len(sb):
        return False
    n = len(sa)
    ok = [[spectra_close(sa[i], sb[j], eps) for j in range(n)] for i in range(n)]
    owner = [-1] * n  # owner[j] = the entry of sa paired with sb[j]

    def augment(i, seen):
        for j in range(n):
            if ok[i][j] and not seen[j]:
                seen[j] = True
                if owner[j] < 0 or augment(owner[j], seen):
                    owner[j] = i
                    return True
        return False

    return all(augment(i, [False] * n) for i in range(n))
