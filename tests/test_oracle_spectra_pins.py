"""Pins of the SVD-invariant oracle (Section 4.2): facts about singular values
that hold independently of how the oracle computes them."""
import itertools

import numpy as np
import pytest

from oracle import spectra as S


def test_masks_cover_each_complement_pair_once():
    for r in range(1, 6):
        ms = S.canonical_masks(r)
        assert len(ms) == (1 << (r - 1)) - 1
        full = (1 << r) - 1
        pairs = {frozenset((g, full ^ g)) for g in range(1, full)}
        assert {frozenset((g, full ^ g)) for g in ms} == pairs


def test_complement_gives_the_same_spectrum():
    rng = np.random.default_rng(1)
    T = rng.standard_normal((3, 4, 5, 2))
    full = 15
    for g in S.canonical_masks(4):
        a = np.linalg.svd(S.unfold(T, g), compute_uv=False)
        b = np.linalg.svd(S.unfold(T, full ^ g), compute_uv=False)
        assert np.allclose(a, b, rtol=0, atol=1e-12 * a[0])


def test_frobenius_norm_of_every_unfolding():
    rng = np.random.default_rng(2)
    T = rng.standard_normal((2, 3, 4, 5, 3))
    fro2 = float(np.sum(T * T))
    for s in S.invariants(T):
        assert abs(float(np.sum(s * s)) - fro2) <= 1e-12 * fro2


def test_rank_one_tensor():
    rng = np.random.default_rng(3)
    vs = [rng.standard_normal(n) for n in (3, 5, 4)]
    T = np.einsum("i,j,k->ijk", *vs)
    norm = np.prod([np.linalg.norm(v) for v in vs])
    for s in S.invariants(T):
        assert abs(s[0] - norm) <= 1e-12 * norm
        assert np.all(s[1:] <= 1e-12 * norm)


def test_orthogonal_unfolding_has_unit_spectrum():
    # a 4x4 Hadamard matrix / 2 is orthogonal; as a 2x2x2x2 tensor, G = {0, 1}
    # is that matrix
    H = np.array([[1, 1, 1, 1], [1, -1, 1, -1], [1, 1, -1, -1], [1, -1, -1, 1]]) / 2.0
    T = H.reshape(2, 2, 2, 2)
    s = S.invariants(T)[S.canonical_masks(4).index(0b0011)]
    assert np.allclose(s, np.ones(4), rtol=0, atol=1e-14)


def test_diagonal_matrix_spectrum_is_sorted_absolute_diagonal():
    d = np.array([3.0, -7.0, 0.5, 2.0])
    (s,) = S.invariants(np.diag(d))
    assert np.array_equal(s, np.sort(np.abs(d))[::-1])


@pytest.mark.parametrize("shape", [(4, 6), (2, 3, 4), (3, 1, 4, 2), (2, 2, 3, 2, 2)])
def test_every_permutation_matches(shape):
    rng = np.random.default_rng(len(shape))
    T = rng.standard_normal(shape).astype(np.float32)
    base = S.invariants(T)
    for perm in itertools.permutations(range(len(shape))):
        assert S.match(base, S.invariants(np.transpose(T, perm)), 1e-10), perm


def test_distinct_tensors_do_not_match():
    rng = np.random.default_rng(9)
    T = rng.standard_normal((3, 4, 5))
    U = T.copy()
    U[1, 2, 3] += 1e-3 * np.abs(T).max()
    assert not S.match(S.invariants(T), S.invariants(U), 1e-6)
    # same values, different grouping of the modes: not a layout change
    assert not S.match(S.invariants(T), S.invariants(T.reshape(4, 3, 5)), 1e-6)
    assert not S.match(S.invariants(T), S.invariants(T.reshape(3, 20)), 1e-6)


def test_pairing_needs_a_search():
    # greedy first-fit pairing fails here; the exhaustive pairing succeeds
    a = [np.array([1.0]), np.array([1.05])]
    b = [np.array([1.04]), np.array([1.0])]
    assert S.match(a, b, 0.045)
    assert not S.match(a, b, 0.001)
