"""Pins for the radius-relation oracle (Section 4.9 generated relation).

Membership is pinned by an independent numpy brute force with the same fp32
predicate, by scipy's cKDTree on binary-grid coordinates whose squared
distances cannot round across the cutoff (the paper's protocol in Section 7.2),
and by symmetry.  Values and gradients are pinned by the sigma -> infinity
special case, by the adjoint identity and by central finite differences.
"""
import numpy as np
import pytest
from scipy.spatial import cKDTree

import oracle
from paper_2609_24802_amd import synth


def brute_neighbours(pos, radius):
    """All ordered pairs (i, j), j != i, with fp32 d2 = (dx*dx + dy*dy) + dz*dz < fp32(r*r)."""
    pos = np.asarray(pos, np.float32)
    r2 = np.float32(radius) * np.float32(radius)
    n = pos.shape[0]
    lists = []
    for i in range(n):
        d = pos - pos[i]  # fp32 direct differences
        d2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
        ok = d2 < r2
        ok[i] = False
        lists.append(np.nonzero(ok)[0])
    return lists


def _lists(ptr, idx):
    return [idx[ptr[k]:ptr[k + 1]] for k in range(len(ptr) - 1)]


@pytest.mark.parametrize("n,radius", [(700, 0.09), (5000, 0.05)])
def test_neighbours_match_brute_force(n, radius):
    # n = 5000 exercises the oracle's cell directory, n = 700 its plain scan
    pos = synth.uniform_f32(n * 3, 0.0, 1.0, (90, n)).reshape(n, 3)
    pos[:5] = pos[5:10]  # coincident distinct points are neighbours
    ptr, idx = oracle.radius_neighbors(pos, radius)
    ref = brute_neighbours(pos, radius)
    for k, lst in enumerate(_lists(ptr, idx)):
        assert np.array_equal(lst, ref[k]), k
    # symmetric relation, even number of directed pairs
    pairs = set(zip(np.repeat(np.arange(n), np.diff(ptr)).tolist(), idx.tolist()))
    assert all((j, i) in pairs for i, j in pairs)
    assert len(pairs) % 2 == 0


def test_binary_grid_matches_kdtree():
    # coordinates are multiples of 2^-6, so squared distances are multiples of 2^-12;
    # r^2 sits strictly between two levels and no rounding can cross it
    pos = synth.binary_grid_points(3000, 6, (91,), span=40)
    r2 = (11.5) * 2.0 ** -12
    radius = np.float32(np.sqrt(r2))
    assert np.float32(radius) * np.float32(radius) > 11 * 2.0 ** -12
    assert np.float32(radius) * np.float32(radius) < 12 * 2.0 ** -12
    ptr, idx = oracle.radius_neighbors(pos, radius)
    tree = cKDTree(pos.astype(np.float64))
    ref = tree.query_ball_point(pos.astype(np.float64), float(radius))
    for k, lst in enumerate(_lists(ptr, idx)):
        exp = np.array(sorted(set(ref[k]) - {k}), dtype=np.int64)
        assert np.array_equal(lst, exp), k


def test_strict_cutoff_rejects_exact_distance():
    # two points exactly r apart (r a power of two) are not neighbours: the test is d2 < r2
    pos = np.array([[0.0, 0.0, 0.0], [0.25, 0.0, 0.0], [0.0, 0.125, 0.0]], np.float32)
    ptr, idx = oracle.radius_neighbors(pos, 0.25)
    assert _lists(ptr, idx)[0].tolist() == [2]
    assert _lists(ptr, idx)[1].tolist() == []


def test_infinite_sigma_is_plain_neighbour_sum():
    n, F = 2000, 3
    pos = synth.uniform_f32(n * 3, 0.0, 1.0, (92,)).reshape(n, 3)
    rng = np.random.default_rng(1)
    x = rng.integers(-5, 6, (n, F)).astype(np.float32)
    y, ya, cnt = oracle.radius_fwd(pos, x, 0.08, 1e30)
    ref = brute_neighbours(pos, 0.08)
    exp = np.stack([x[l].astype(np.float64).sum(0) for l in ref])
    assert np.array_equal(y, exp)
    assert np.array_equal(cnt, [len(l) for l in ref])


def test_weights_against_explicit_pairs():
    n, F = 400, 4
    pos = synth.uniform_f32(n * 3, 0.0, 1.0, (93,)).reshape(n, 3)
    x = synth.normal_f32(n * F, (93, 1)).reshape(n, F)
    r, s = np.float32(0.2), np.float32(0.1)
    y, ya, cnt = oracle.radius_fwd(pos, x, r, s)
    ref = brute_neighbours(pos, r)
    p64 = pos.astype(np.float64)
    for i in range(0, n, 37):
        d2 = ((p64[ref[i]] - p64[i]) ** 2).sum(1)
        k = np.exp(-d2 / (float(s) ** 2))
        np.testing.assert_allclose(y[i], k @ x[ref[i]].astype(np.float64), rtol=1e-12, atol=1e-14)
    # subset evaluation returns the same rows
    pts = np.array([5, 399, 0, 5])
    ys, _, cs = oracle.radius_fwd(pos, x, r, s, pts=pts)
    assert np.array_equal(ys, y[pts]) and np.array_equal(cs, cnt[pts])


def _fd_points(seed):
    """32 points in a unit box with every pair distance at least 1e-3 away from the cutoff."""
    r = 0.45
    for s in range(seed, seed + 200):
        pos = synth.uniform_f32(32 * 3, 0.0, 1.0, (94, s)).reshape(32, 3)
        d = np.sqrt(((pos[:, None, :].astype(np.float64) - pos[None]) ** 2).sum(-1))
        if np.abs(d - r).min() > 1e-3:
            return pos, np.float32(r)
    raise RuntimeError("no admissible configuration")


def test_backward_finite_differences():
    pos, r = _fd_points(0)
    n, F = pos.shape[0], 3
    sigma = np.float32(0.3)
    x = synth.normal_f32(n * F, (95, 1)).reshape(n, F)
    dy = synth.normal_f32(n * F, (95, 2)).reshape(n, F)
    dx, _, dp, _ = oracle.radius_bwd(pos, x, dy, r, sigma)

    def loss(pp, xx):
        y, _, _ = oracle.radius_fwd(pp, xx, r, sigma)
        return float((y * dy).sum())

    # the forward is linear in x: <y, dy> = <x, dx>
    np.testing.assert_allclose(loss(pos, x), float((x * dx).sum()), rtol=1e-12)
    h = np.float32(2.0 ** -14)
    for i, a in [(0, 0), (3, 1), (10, 2), (31, 0), (17, 1)]:
        pp, pm = pos.copy(), pos.copy()
        pp[i, a] += h
        pm[i, a] -= h
        fd = (loss(pp, x) - loss(pm, x)) / (float(pp[i, a]) - float(pm[i, a]))
        assert abs(fd - dp[i, a]) <= 2e-6 * (1 + abs(fd)), (i, a, fd, dp[i, a])
    for i, f in [(1, 0), (20, 2)]:
        xp, xm = x.copy(), x.copy()
        xp[i, f] += h
        xm[i, f] -= h
        fd = (loss(pos, xp) - loss(pos, xm)) / (float(xp[i, f]) - float(xm[i, f]))
        assert abs(fd - dx[i, f]) <= 1e-8 * (1 + abs(fd))


def test_backward_subset_and_grid_path():
    n, F = 6000, 2
    pos = synth.uniform_f32(n * 3, 0.0, 1.0, (96,)).reshape(n, 3)
    x = synth.normal_f32(n * F, (96, 1)).reshape(n, F)
    dy = synth.normal_f32(n * F, (96, 2)).reshape(n, F)
    r, s = np.float32(0.06), np.float32(0.03)
    dx, _, dp, _ = oracle.radius_bwd(pos, x, dy, r, s)
    pts = np.array([0, 4321, 5999])
    dxs, _, dps, _ = oracle.radius_bwd(pos, x, dy, r, s, pts=pts)
    assert np.array_equal(dxs, dx[pts]) and np.array_equal(dps, dp[pts])
    # translation invariance: the position gradients sum to zero
    np.testing.assert_allclose(dp.sum(0), 0.0, atol=1e-9 * np.abs(dp).sum())
    y, _, _ = oracle.radius_fwd(pos, x, r, s)
    np.testing.assert_allclose(float((y * dy).sum()), float((x * dx).sum()), rtol=1e-11)


def test_config3_radius_constant_and_mean_degree():
    r = synth.radius_for_mean_degree(1_000_000)
    assert abs(float(r) - 0.0196949) < 1e-6
    # a smaller cloud with the same expected degree: interior mean close to 32
    n = 200_000
    pos = synth.uniform_f32(n * 3, 0.0, 1.0, (97,)).reshape(n, 3)
    rn = synth.radius_for_mean_degree(n)
    inner = np.nonzero(np.all((pos > 2 * rn) & (pos < 1 - 2 * rn), axis=1))[0][:4000]
    _, _, cnt = oracle.radius_fwd(pos, np.zeros((n, 1), np.float32), rn, rn / 2, pts=inner)
    assert abs(cnt.mean() - 32.0) < 0.6


def _corner_cloud(n, seed):
    """A cloud whose point 0 lies below every other point in all three coordinates and whose last
    point lies above every other point, inside one radius of each other."""
    pos = synth.uniform_f32(n * 3, 0.2, 0.3, (98, n, seed)).reshape(n, 3)
    pos[0] = 0.19
    pos[-1] = 0.31
    return pos


@pytest.mark.parametrize("n", [300, 4500])
def test_sum_of_term_magnitudes_is_exact_without_cancellation(n):
    """Each output's sum|terms| equals the output itself when no term can be negative: y with x >= 0,
    dx with dy >= 0, and the position gradient of a point below (above) all of its neighbours, whose
    displacements are all >= 0 (<= 0), with x and dy positive.  n = 4500 takes the cell directory."""
    pos = _corner_cloud(n, 1)
    F = 3
    x = synth.uniform_f32(n * F, 0.5, 1.5, (99, n, 1)).reshape(n, F)
    dy = synth.uniform_f32(n * F, 0.5, 1.5, (99, n, 2)).reshape(n, F)
    r, s = np.float32(0.2), np.float32(0.05)
    y, ya, cnt = oracle.radius_fwd(pos, x, r, s)
    assert np.array_equal(ya, y) and cnt.min() > 0
    dx, dxa, dp, dpa = oracle.radius_bwd(pos, x, dy, r, s)
    assert np.array_equal(dxa, dx)
    assert np.all(dp[0] > 0) and np.array_equal(dpa[0], dp[0])
    assert np.all(dp[-1] < 0) and np.array_equal(dpa[-1], -dp[-1])
    # with mixed signs the magnitudes bound the values and exceed them somewhere
    xm = synth.normal_f32(n * F, (99, n, 3)).reshape(n, F)
    dym = synth.normal_f32(n * F, (99, n, 4)).reshape(n, F)
    y, ya, _ = oracle.radius_fwd(pos, xm, r, s)
    dx, dxa, dp, dpa = oracle.radius_bwd(pos, xm, dym, r, s)
    for v, m in ((y, ya), (dx, dxa), (dp, dpa)):
        assert np.all(np.abs(v) <= m * (1 + 1e-15)) and (m > np.abs(v) * (1 + 1e-9)).any()


def test_position_gradient_magnitude_two_points():
    """Two neighbours: dp_0 = (2k/sigma^2) d (<dy_0, x_1> + <dy_1, x_0>) with d = p_1 - p_0 >= 0, so
    with positive features its magnitude is dp_0 and that of dp_1 is -dp_1 = dp_0."""
    pos = np.array([[0.1, 0.2, 0.3], [0.125, 0.25, 0.3125]], np.float32)
    x = np.array([[1.0, 2.0], [0.5, 3.0]], np.float32)
    dy = np.array([[2.0, 1.0], [1.0, 0.25]], np.float32)
    r, s = np.float32(0.5), np.float32(0.25)
    dx, dxa, dp, dpa = oracle.radius_bwd(pos, x, dy, r, s)
    d = pos[1].astype(np.float64) - pos[0]
    k = np.exp(-(d @ d) / float(s) ** 2)
    inner = float(dy[0] @ x[1] + dy[1] @ x[0])
    np.testing.assert_allclose(dp[0], 2 * k / float(s) ** 2 * d * inner, rtol=1e-14)
    assert np.array_equal(dpa[0], dp[0]) and np.array_equal(dpa[1], -dp[1])
    assert np.array_equal(dp[1], -dp[0])
    # mixed signs: the inner products' four terms enter with their absolute values
    dy = np.array([[2.0, -1.0], [-1.0, 0.25]], np.float32)
    x = np.array([[1.0, -2.0], [0.5, 3.0]], np.float32)
    dx, dxa, dp, dpa = oracle.radius_bwd(pos, x, dy, r, s)
    absinner = float(np.abs(dy[0]) @ np.abs(x[1]) + np.abs(dy[1]) @ np.abs(x[0]))
    np.testing.assert_allclose(dpa[0], 2 * k / float(s) ** 2 * d * absinner, rtol=1e-14)
    np.testing.assert_allclose(dpa[1], dpa[0], rtol=1e-14)
    np.testing.assert_allclose(dxa, k * np.abs(dy[::-1]), rtol=1e-14)


def test_config3_cloud_against_kdtree():
    """The paper's edge-set protocol on the measured cloud itself (1M points): the oracle's relation
    equals scipy's fp64 ball query (distance <= r), except for pairs whose fp64 squared distance lies
    within 4 fp32 ulp of r^2, where fp32 rounding may decide either way."""
    g = synth.config3()
    pos, r = g["pos"], g["radius"]
    n = pos.shape[0]
    ptr, idx = oracle.radius_neighbors(pos, r)
    src = np.repeat(np.arange(n, dtype=np.int64), np.diff(ptr))
    up = src < idx
    assert 2 * int(up.sum()) == int(ptr[-1])            # symmetric: each pair listed both ways
    mine = src[up] * n + idx[up]
    tree = cKDTree(pos.astype(np.float64))
    pairs = tree.query_pairs(float(r), output_type="ndarray").astype(np.int64)
    ref = pairs.min(1) * n + pairs.max(1)
    diff = np.setxor1d(mine, ref)
    assert diff.size < 50
    i, j = diff // n, diff % n
    d = pos[j].astype(np.float64) - pos[i]
    d2 = (d * d).sum(1)
    r2 = float(np.float32(r) * np.float32(r))
    ulp = float(np.spacing(np.float32(r2)))
    assert np.all(np.abs(d2 - r2) <= 4 * ulp), np.abs(d2 - r2).max() / ulp
