"""Pins for the CSR oracle (weighted sum and max, forward and VJP).

Each test checks the oracle against something other than itself: the worked
example printed in Section 3.1, scipy.sparse and torch library routines,
invariants of the weighted sum, and central finite differences.
"""
import json
import os

import numpy as np
import pytest
import scipy.sparse as sp
import torch

import oracle
from paper_2609_24802_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def _graph(num_dst, num_src, num_edges, F, seed, empty_rows=True, integer=False):
    """Random multigraph with duplicates, self-loops (when square) and empty rows."""
    rng = np.random.default_rng(seed)
    dst = rng.integers(0, num_dst, num_edges)
    if empty_rows:
        dst = np.where(dst % 7 == 3, (dst + 1) % num_dst, dst)  # rows = 3 mod 7 stay empty
    src = rng.integers(0, num_src, num_edges)
    src[: num_edges // 10] = src[num_edges // 10: 2 * (num_edges // 10)]  # duplicates
    order = np.argsort(dst, kind="stable")
    dst, src = dst[order], src[order]
    row_ptr = np.zeros(num_dst + 1, np.int64)
    np.cumsum(np.bincount(dst, minlength=num_dst), out=row_ptr[1:])
    if integer:
        x = rng.integers(-4, 5, (num_src, F)).astype(np.float32)
        w = rng.integers(0, 4, num_edges).astype(np.float32)
        dy = rng.integers(-3, 4, (num_dst, F)).astype(np.float32)
    else:
        x = rng.standard_normal((num_src, F)).astype(np.float32)
        w = rng.random(num_edges).astype(np.float32)
        dy = rng.standard_normal((num_dst, F)).astype(np.float32)
    return row_ptr, src.astype(np.int32), dst, x, w, dy


def test_worked_example_sum():
    g = json.load(open(GOLD))
    rp, col = np.array(g["row_ptr"]), np.array(g["col_idx"])
    x = np.array(g["x"], np.float32)[:, None]
    w = np.array(g["w"], np.float32)
    dy = np.array(g["dy"], np.float32)[:, None]
    y, _ = oracle.csr_sum_fwd(rp, col, x, w)
    assert y[:, 0].tolist() == g["printed"]["y"]
    dx, _, dw, _ = oracle.csr_sum_bwd(rp, col, x, w, dy, g["num_src"])
    assert dx[:, 0].tolist() == g["printed"]["dx"]
    assert dw.tolist() == g["printed"]["dw"]


def test_worked_example_max():
    g = json.load(open(GOLD))
    rp, col = np.array(g["row_ptr"]), np.array(g["col_idx"])
    x = np.array(g["x"], np.float32)[:, None]
    w = np.array(g["w"], np.float32)
    dy = np.array(g["dy"], np.float32)[:, None]
    y, arg = oracle.csr_max_fwd(rp, col, x, w)
    d = g["derived_max"]
    assert y[:, 0].tolist() == d["y"] and arg[:, 0].tolist() == d["arg"]
    dx, _, dw, _ = oracle.csr_max_bwd(rp, col, x, w, arg, dy, g["num_src"])
    assert dx[:, 0].tolist() == d["dx"] and dw.tolist() == d["dw"]


@pytest.mark.parametrize("num_dst,num_src,F", [(300, 300, 1), (257, 131, 5), (64, 500, 16)])
def test_sum_matches_scipy(num_dst, num_src, F):
    rp, col, dst, x, w, dy = _graph(num_dst, num_src, 4000, F, seed=F)
    A = sp.csr_matrix((w.astype(np.float64), col, rp), shape=(num_dst, num_src))
    y, ya = oracle.csr_sum_fwd(rp, col, x, w)
    np.testing.assert_allclose(y, A @ x.astype(np.float64), rtol=1e-12, atol=1e-12)
    dx, _, dw, _ = oracle.csr_sum_bwd(rp, col, x, w, dy, num_src)
    np.testing.assert_allclose(dx, A.T @ dy.astype(np.float64), rtol=1e-12, atol=1e-12)
    # SDDMM through a dense product sampled at the pattern: dw_e = (dy x^T)[d(e), s(e)]
    dense = dy.astype(np.float64) @ x.astype(np.float64).T
    np.testing.assert_allclose(dw, dense[dst, col], rtol=1e-12, atol=1e-12)
    # unweighted message (w = 1) is the pattern matrix
    y1, _ = oracle.csr_sum_fwd(rp, col, x, None)
    P = sp.csr_matrix((np.ones_like(w, np.float64), col, rp), shape=(num_dst, num_src))
    np.testing.assert_allclose(y1, P @ x.astype(np.float64), rtol=1e-12, atol=1e-12)
    assert np.all(ya >= np.abs(y) - 1e-12)


def test_sum_invariants_and_adjoint():
    rp, col, dst, x, w, dy = _graph(500, 400, 6000, 3, seed=11)
    y, _ = oracle.csr_sum_fwd(rp, col, x, w)
    # total of all outputs equals the total of all per-edge messages
    out_w = np.bincount(col, weights=w.astype(np.float64), minlength=400)
    np.testing.assert_allclose(y.sum(0), out_w @ x.astype(np.float64), rtol=1e-12)
    # empty rows finalize to the sum identity
    empty = np.diff(rp) == 0
    assert empty.any() and np.all(y[empty] == 0.0)
    # degrees are the row-pointer differences
    assert np.array_equal(np.diff(rp), np.bincount(dst, minlength=500))
    # bilinearity: <y, dy> = <x, dx> = <w, dw>
    dx, _, dw, _ = oracle.csr_sum_bwd(rp, col, x, w, dy, 400)
    a = float((y * dy).sum())
    np.testing.assert_allclose(a, float((x * dx).sum()), rtol=1e-11)
    np.testing.assert_allclose(a, float((w * dw).sum()), rtol=1e-11)


def test_sum_finite_differences():
    rp, col, dst, x, w, dy = _graph(20, 15, 90, 2, seed=5)
    dx, _, dw, _ = oracle.csr_sum_bwd(rp, col, x, w, dy, 15)

    def loss(xx, ww):
        y, _ = oracle.csr_sum_fwd(rp, col, xx, ww)
        return float((y * dy).sum())

    h = np.float32(2.0 ** -10)
    for j, f in [(0, 0), (3, 1), (7, 0), (14, 1)]:
        xp, xm = x.copy(), x.copy()
        xp[j, f] += h
        xm[j, f] -= h
        fd = (loss(xp, w) - loss(xm, w)) / (float(xp[j, f]) - float(xm[j, f]))
        assert abs(fd - dx[j, f]) <= 1e-9 * (1 + abs(fd))
    for e in [0, 17, 45, 89]:
        wp, wm = w.copy(), w.copy()
        wp[e] += h
        wm[e] -= h
        fd = (loss(x, wp) - loss(x, wm)) / (float(wp[e]) - float(wm[e]))
        assert abs(fd - dw[e]) <= 1e-9 * (1 + abs(fd))


def test_max_matches_torch_and_argmax():
    rp, col, dst, x, w, dy = _graph(300, 200, 5000, 4, seed=3)
    y, arg = oracle.csr_max_fwd(rp, col, x, w)
    msg = torch.from_numpy(w)[:, None] * torch.from_numpy(x)[torch.from_numpy(col).long()]
    ref = torch.zeros(300, 4).scatter_reduce(0, torch.from_numpy(dst)[:, None].expand(-1, 4), msg,
                                             "amax", include_self=False)
    nonempty = np.diff(rp) > 0
    assert np.array_equal(y[nonempty], ref.numpy()[nonempty])
    assert np.all(y[~nonempty] == 0) and np.all(arg[~nonempty] == -1)
    # argmax is the first position attaining the maximum (numpy's argmax rule)
    m = msg.numpy()
    for i in np.nonzero(nonempty)[0]:
        lo, hi = rp[i], rp[i + 1]
        assert np.array_equal(arg[i], lo + np.argmax(m[lo:hi], axis=0))


def test_max_constructed_ties():
    # duplicate edges with equal weight: every tie goes to the lowest position
    rp = np.array([0, 4, 6, 6, 9])
    col = np.array([2, 2, 1, 2, 0, 0, 1, 1, 1], np.int32)
    x = np.array([[1.0, -2.0], [3.0, 0.0], [3.0, 5.0]], np.float32)
    w = np.array([1, 1, 1, 1, 2, 2, 0.5, 0.5, 0.5], np.float32)
    y, arg = oracle.csr_max_fwd(rp, col, x, w)
    assert arg.tolist() == [[0, 0], [4, 4], [-1, -1], [6, 6]]
    assert y.tolist() == [[3.0, 5.0], [2.0, -4.0], [0.0, 0.0], [1.5, 0.0]]
    # all-zero features: every message is 0 and the first edge wins
    y0, a0 = oracle.csr_max_fwd(rp, col, np.zeros_like(x), w)
    assert a0[:, 0].tolist() == [0, 4, -1, 6] and np.all(y0 == 0)
    # -0 and +0 tie: the first edge's value (and sign bit) is kept
    xs = np.array([[-1.0], [1.0]], np.float32)
    ys, as_ = oracle.csr_max_fwd(np.array([0, 2]), np.array([0, 1], np.int32), xs,
                                 np.array([0.0, 0.0], np.float32))
    assert as_[0, 0] == 0 and np.signbit(ys[0, 0])


def test_max_backward_matches_torch_autograd():
    rp, col, dst, x, w, dy = _graph(150, 120, 2500, 3, seed=9)
    y, arg = oracle.csr_max_fwd(rp, col, x, w)
    xt = torch.from_numpy(x.astype(np.float64)).requires_grad_()
    wt = torch.from_numpy(w.astype(np.float64)).requires_grad_()
    msg = wt[:, None] * xt[torch.from_numpy(col).long()]
    out = torch.zeros(150, 3, dtype=torch.float64).scatter_reduce(
        0, torch.from_numpy(dst)[:, None].expand(-1, 3), msg, "amax", include_self=False)
    gx, gw = torch.autograd.grad(out, (xt, wt), torch.from_numpy(dy.astype(np.float64)))
    dx, _, dw, _ = oracle.csr_max_bwd(rp, col, x, w, arg, dy, 120)
    # random continuous inputs have no ties, where torch's amax gradient is the routed one
    np.testing.assert_allclose(dx, gx.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, gw.numpy(), rtol=1e-12, atol=1e-12)
    a = float((y.astype(np.float64) * dy).sum())
    np.testing.assert_allclose(a, float((x * dx).sum()), rtol=1e-6)
    np.testing.assert_allclose(a, float((w * dw).sum()), rtol=1e-6)


def test_row_subset_and_integer_exactness():
    rp, col, dst, x, w, dy = _graph(400, 400, 7000, 6, seed=21, integer=True)
    y, ya = oracle.csr_sum_fwd(rp, col, x, w)
    rows = np.array([399, 0, 17, 17, 250])
    ys, yas = oracle.csr_sum_fwd(rp, col, x, w, rows=rows)
    assert np.array_equal(ys, y[rows]) and np.array_equal(yas, ya[rows])
    assert np.all(y == np.round(y))
    ym, am = oracle.csr_max_fwd(rp, col, x, w)
    yms, ams = oracle.csr_max_fwd(rp, col, x, w, rows=rows)
    assert np.array_equal(yms, ym[rows]) and np.array_equal(ams, am[rows])


def test_powerlaw_generator_shapes():
    g = synth.config2(scale=0.002)
    rp, col = g["row_ptr"], g["col"]
    n = g["num_dst"]
    assert rp[0] == 0 and rp[-1] == col.shape[0] == 16 * n
    assert np.all(np.diff(rp) >= 0) and col.min() >= 0 and col.max() < n
    y, _ = oracle.csr_sum_fwd(rp, col, g["x"], g["w"], rows=np.arange(10))
    A = sp.csr_matrix((g["w"].astype(np.float64), col, rp), shape=(n, n))
    np.testing.assert_allclose(y, (A @ g["x"].astype(np.float64))[:10], rtol=1e-12, atol=1e-12)


def test_results_do_not_depend_on_thread_count():
    """Each output is summed by one thread in a fixed order, so one thread and all host threads give
    the same bits (the baseline timing runs both)."""
    g = synth.csr_uniform_small()
    args = (g["row_ptr"], g["col"], g["x"], g["w"])
    try:
        oracle.set_threads(1)
        one = oracle.csr_sum_fwd(*args), oracle.csr_sum_bwd(*args, g["dy"], g["num_src"])
    finally:
        oracle.set_threads(0)
    many = oracle.csr_sum_fwd(*args), oracle.csr_sum_bwd(*args, g["dy"], g["num_src"])
    for a, b in zip(one, many):
        for u, v in zip(a, b):
            assert np.array_equal(u, v)
