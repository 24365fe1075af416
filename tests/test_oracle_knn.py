"""Pins for the oracle's exact kNN relation (the generated kNN of Section 4.9 and its Section 7 workload).

Checks come from outside the oracle's own selection loop: a hand-derived closed form on a line
(distance ties resolved by index), numpy's lexsort over the same fp32 squared distances, the
k = n - 1 special case, coincident points, and invariances (relabeling, exact translation)."""
import numpy as np
import pytest

import oracle
from paper_2609_24802_amd import synth


def d2_f32(pos):
    """The fp32 squared-distance recipe, written with numpy float32 arithmetic (no contraction)."""
    p = pos.astype(np.float32)
    dx = p[None, :, 0] - p[:, None, 0]
    dy = p[None, :, 1] - p[:, None, 1]
    dz = p[None, :, 2] - p[:, None, 2]
    return (dx * dx + dy * dy) + dz * dz


def test_line_closed_form():
    """Points at 0, 1, ..., n-1 on the x axis: query i takes i-1, i+1, i-2, i+2, ... (the lower
    index first at each distance), skipping indices outside [0, n)."""
    n, k = 23, 7
    pos = np.zeros((n, 3), np.float32)
    pos[:, 0] = np.arange(n)
    nbr, y, _ = oracle.knn(pos, np.arange(n, dtype=np.float32)[:, None] ** 2, k)
    for i in range(n):
        want = []
        for dist in range(1, n):
            for j in (i - dist, i + dist):
                if 0 <= j < n and len(want) < k:
                    want.append(j)
        assert list(nbr[i]) == want, (i, nbr[i], want)
        assert y[i, 0] == sum(j * j for j in want)


@pytest.mark.parametrize("n,k,seed", [(50, 1, 0), (97, 5, 1), (200, 16, 2), (64, 32, 3), (33, 31, 4)])
def test_brute_force_lexsort(n, k, seed):
    rng = np.random.default_rng(seed)
    pos = rng.random((n, 3), dtype=np.float32)
    x = rng.standard_normal((n, 3)).astype(np.float32)
    nbr, y, ya = oracle.knn(pos, x, k)
    d2 = d2_f32(pos)
    idx = np.arange(n)
    for i in range(n):
        j = idx[idx != i]
        order = np.lexsort((j, d2[i, j]))        # primary key d2, then index
        sel = j[order[:k]]
        assert np.array_equal(nbr[i], sel)
        np.testing.assert_allclose(y[i], x[sel].astype(np.float64).sum(0), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(ya[i], np.abs(x[sel].astype(np.float64)).sum(0), rtol=1e-12)


def test_all_others_when_k_is_n_minus_one():
    n = 40
    pos = synth.uniform_f32(n * 3, 0.0, 1.0, (90, 0)).reshape(n, 3)
    x = synth.normal_f32(n * 2, (90, 1)).reshape(n, 2)
    nbr, y, _ = oracle.knn(pos, x, n - 1)
    tot = x.astype(np.float64).sum(0)
    for i in range(n):
        assert sorted(nbr[i]) == [j for j in range(n) if j != i]
        np.testing.assert_allclose(y[i], tot - x[i], rtol=1e-12, atol=1e-12)


def test_coincident_points_rank_by_index():
    """Five copies of one point and a far cloud: each copy selects the other copies first, in index
    order (all at d2 = 0), then the nearest far points."""
    rng = np.random.default_rng(7)
    pos = (rng.random((30, 3)) * 10 + 5).astype(np.float32)
    copies = [3, 8, 11, 20, 27]
    pos[copies] = np.float32(0.25)
    nbr, _, _ = oracle.knn(pos, None, 6)
    for c in copies:
        assert list(nbr[c][:4]) == [j for j in copies if j != c]


def test_relabeling_is_equivariant():
    rng = np.random.default_rng(11)
    n, k = 120, 8
    pos = rng.random((n, 3), dtype=np.float32)
    x = rng.standard_normal((n, 1)).astype(np.float32)
    perm = rng.permutation(n)
    nbr, y, _ = oracle.knn(pos, x, k)
    nbr_p, y_p, _ = oracle.knn(pos[perm], x[perm], k)
    # random coordinates: no distance ties, so the selected sets map through the permutation
    for a in range(n):
        assert sorted(perm[nbr_p[a]]) == sorted(nbr[perm[a]])
        np.testing.assert_allclose(y_p[a], y[perm[a]], rtol=1e-12)


def test_exact_translation_on_binary_grid():
    pos = synth.binary_grid_points(300, 6, (91, 0), span=40)
    shifted = (pos + np.float32(3.0)).astype(np.float32)     # exact: multiples of 2^-6 below 2^2
    assert np.array_equal(shifted - np.float32(3.0), pos)
    a, _, _ = oracle.knn(pos, None, 12)
    b, _, _ = oracle.knn(shifted, None, 12)
    assert np.array_equal(a, b)


def test_non_finite_points_are_never_selected():
    rng = np.random.default_rng(5)
    pos = rng.random((20, 3), dtype=np.float32)
    pos[4, 1] = np.nan
    pos[9, 0] = np.inf
    nbr, y, _ = oracle.knn(pos, np.ones((20, 1), np.float32), 19)
    for i in range(20):
        if i in (4, 9):
            assert (nbr[i] == -1).all() and y[i, 0] == 0.0     # no finite distance from here
        else:
            assert 4 not in nbr[i] and 9 not in nbr[i]
            assert (nbr[i][:17] >= 0).all() and (nbr[i][17:] == -1).all()
            assert y[i, 0] == 17.0
