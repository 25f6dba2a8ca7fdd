"""Multi-mode SVD invariants and tensor matching (Section 4.2) on the GPU,
through the C ABI, against the oracle.

Spectra: every eigenvalue sigma^2 within 1e-9 of the unfolding's largest
(the fp64 Gram sums at most a few million fp32 products, each exact, and the
tridiagonal reduction and bisection are backward stable, so the error is far
below that).  Matching: the GPU's decisions equal the oracle's on the same
spectra, and planted permutations match while perturbed tensors do not.
"""
import itertools

import numpy as np
import pytest

from gpu_util import log
from oracle import spectra as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2512_08365_amd as mag
    mag.version()
    yield


def _gpu_lists(arrays):
    import torch
    import paper_2512_08365_amd as mag
    ts = [torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda() for a in arrays]
    spec, lay = mag.invariants(ts)
    flat = spec.cpu().numpy()
    out, o = [], 0
    for lens in lay:
        lst = []
        for n in lens:
            lst.append(flat[o:o + n])
            o += n
        out.append(lst)
    assert o == flat.size
    return ts, spec, out


def _assert_spectra(got, want, label):
    assert len(got) == len(want), label
    for g, w in zip(got, want):
        assert g.shape == w.shape, label
        top = max(float(w[0]), 1e-300) ** 2
        err = np.abs(g.astype(np.float64) ** 2 - w ** 2).max()
        assert err <= 1e-9 * top, (label, err / top)
        assert np.all(np.diff(g) <= 0), label  # descending


SHAPES = [(5,), (1, 1), (3, 7), (16, 16), (17, 33), (2, 3, 4), (4, 1, 9), (8, 64, 128),
          (3, 5, 2, 7), (2, 3, 2, 3, 2), (1, 4, 1, 5, 1), (100, 600), (511, 40), (512, 512),
          (2, 256, 4096), (20, 25, 700),
          # Gram sides in (64, 128], each made by one workgroup per column
          # chunk: just above 64, ragged column chunks and steps, rows from two
          # modes, both gather directions of the attention-shaped tensors
          (65, 3000), (3, 40, 1100), (128, 2049), (32, 128, 128),
          # Gram sides above 512: the many-workgroup reduction (one or two large
          # unfoldings beside a small one, a side not a multiple of the blocks)
          (600, 700), (2, 600, 700), (1030, 1100)]


@pytest.mark.parametrize("shape", SHAPES)
def test_spectra_match_the_oracle(shape):
    rng = np.random.default_rng(sum(shape))
    T = rng.standard_normal(shape).astype(np.float32)
    if len(shape) >= 2:
        T[..., 0] *= 50.0  # a spread of singular values
    log(f"[spectra] shape {shape}")
    _, _, (got,) = _gpu_lists([T])
    _assert_spectra(got, S.invariants(T), f"{shape}")


def test_closed_forms_on_the_gpu():
    rng = np.random.default_rng(4)
    vs = [rng.standard_normal(n).astype(np.float32) for n in (6, 9, 5)]
    R1 = np.einsum("i,j,k->ijk", *vs)
    H = np.array([[1, 1, 1, 1], [1, -1, 1, -1], [1, 1, -1, -1], [1, -1, -1, 1]], np.float32) / 2
    _, _, (r1, h) = _gpu_lists([R1, H.reshape(2, 2, 2, 2)])
    norm = float(np.prod([np.linalg.norm(v.astype(np.float64)) for v in vs]))
    for s in r1:
        assert abs(s[0] - norm) <= 1e-6 * norm and np.all(s[1:] <= 1e-6 * norm)
    assert np.allclose(h[S.canonical_masks(4).index(0b0011)], 1.0, atol=1e-7)


@pytest.mark.parametrize("k,l", [(128, 600), (96, 257)])
def test_clustered_spectra_whole_triangle_sides(k, l):
    """Gram sides in (64, 128] (one workgroup per column chunk makes the whole
    triangle) with repeated and clustered singular values, where bisection
    has to separate equal eigenvalues: against the oracle on the same fp32
    data, and against the singular values the matrix was built from (its
    fp32 rounding moves them by about 1e-7 relative)."""
    rng = np.random.default_rng(k + l)
    q = rng.standard_normal((k, k))
    u, _ = np.linalg.qr(q)
    w, _ = np.linalg.qr(rng.standard_normal((l, k)))
    parts = [np.full(k // 6, 10.0), np.full(k // 4, 5.0), 1.0 + 1e-6 * np.arange(k // 6),
             np.linspace(1.5, 3.0, k // 6)]
    sv = np.concatenate(parts)
    sv = np.concatenate([sv, np.full(k - sv.size, 1e-3)])
    X = ((u * sv) @ w.T).astype(np.float32)
    log(f"[spectra] clustered {k} x {l}")
    _, _, (got,) = _gpu_lists([X])
    _assert_spectra(got, S.invariants(X), f"clustered {k} x {l}")
    want = np.sort(sv)[::-1]
    assert np.abs(got[0].astype(np.float64) - want).max() <= 1e-5 * want[0]


def test_mixed_batch_in_one_call():
    """One call over tensors of every Gram class (one 32-side block, the whole
    triangle for sides in (64, 128], 64-side blocks, and sides above 512 on
    the many-workgroup path), so the library's reordering of the unfoldings
    by class and its numbering of the eigenvalue work items (large sides have
    none) are checked against each tensor's own oracle lists, in input order."""
    rng = np.random.default_rng(21)
    shapes = [(5,), (100, 600), (600, 700), (3, 40, 1100), (17, 33), (2, 256, 4096), (65, 80),
              (8, 64, 128), (1, 1)]
    Ts = [rng.standard_normal(sh).astype(np.float32) for sh in shapes]
    log(f"[spectra] mixed batch {shapes}")
    _, _, got = _gpu_lists(Ts)
    assert len(got) == len(Ts)
    for T, g, sh in zip(Ts, got, shapes):
        _assert_spectra(g, S.invariants(T), f"mixed {sh}")


def test_matching_planted_permutations():
    rng = np.random.default_rng(11)
    A = [rng.standard_normal(s).astype(np.float32) for s in
         [(4, 6, 5), (3, 3, 8), (2, 5, 2, 3), (30, 20), (6, 8, 10)]]
    B = []
    truth = np.zeros((len(A), 0), bool)
    cols = []
    for i, a in enumerate(A):
        perm = tuple(rng.permutation(a.ndim))
        B.append(np.ascontiguousarray(np.transpose(a, perm)))  # a layout change: matches
        cols.append(i)
        bad = a.copy()
        bad.flat[7] += 1e-2 * np.abs(a).max()  # a different tensor: does not
        B.append(bad)
        cols.append(-1)
    B.append(A[0].reshape(6, 4, 5).copy())  # regrouped modes: not a layout change
    cols.append(-1)
    import paper_2512_08365_amd as mag
    ta, sa, la = _gpu_lists(A)
    tb, sb, lb = _gpu_lists(B)
    got = mag.match(ta, sa, tb, sb, 1e-5).cpu().numpy()
    want = np.array([[S.match(x, y, 1e-5) for y in lb] for x in la], np.uint8)
    assert np.array_equal(got, want)  # the same decisions on the same spectra
    planted = np.array([[c == i for c in cols] for i in range(len(A))], np.uint8)
    assert np.array_equal(got, planted), (got, planted)


@pytest.mark.parametrize("shape", [(3, 4, 5, 2)])
def test_every_permutation_matches_on_the_gpu(shape):
    import paper_2512_08365_amd as mag
    rng = np.random.default_rng(5)
    T = rng.standard_normal(shape).astype(np.float32)
    perms = [np.ascontiguousarray(np.transpose(T, p)) for p in itertools.permutations(range(4))]
    ta, sa, _ = _gpu_lists([T])
    tb, sb, _ = _gpu_lists(perms)
    assert mag.match(ta, sa, tb, sb, 1e-5).cpu().numpy().all()


def test_unsupported_shapes_are_rejected():
    import torch
    import paper_2512_08365_amd as mag
    with pytest.raises(mag.MagnetonError) as e:
        # min(M, N) = 8193 > MAG_SVD_MAX_K (refused before any device work)
        mag.invariants([torch.empty((8193, 8194), device="cuda")])
    assert e.value.code == -2
    with pytest.raises(mag.MagnetonError):
        mag.invariants([torch.zeros((2,) * 6, device="cuda")])  # rank 6


def test_large_rank_deficient_unfolding():
    """A Gram side above 512 whose matrix is rank-deficient (zero rows, and
    rows repeated): Householder steps whose column is already reduced are
    skipped, and the zero eigenvalues come out within the bound."""
    rng = np.random.default_rng(12)
    T = np.zeros((700, 800), np.float32)
    T[:300] = rng.standard_normal((300, 800)).astype(np.float32)
    T[300:350] = T[:50]  # repeated rows
    T[:, :3] *= 40.0
    log("[spectra] rank-deficient 700 x 800")
    _, _, (got,) = _gpu_lists([T])
    _assert_spectra(got, S.invariants(T), "rank-deficient 700 x 800")
