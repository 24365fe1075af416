"""Pins for the oracle's edge-local MLP message (the EdgeNN appendix) and its vector-Jacobian product.

The network is piecewise linear in every input and parameter, and the loss <dy, y> is at most linear
in any single coordinate (W2 multiplies ReLU outputs that do not depend on W2), so central
differences of the forward are exact up to fp64 rounding away from ReLU kinks: they pin every
gradient.  Closed forms pin the forward (all units active: an affine map of summed inputs; W2 = 0:
only the final bias, once per neighbour)."""
import numpy as np
import pytest

import oracle
from paper_2609_24802_amd import synth


def relation(pos, r):
    return oracle.radius_neighbors(pos, r)


def small_case(seed, n=24, F=2, H=5, O=2):
    rng = np.random.default_rng(seed)
    # multiples of 2^-8 so that +-2^-12 perturbations stay exact in fp32
    pos = (rng.integers(0, 64, (n, 3)) / 256.0).astype(np.float32)
    x = (rng.integers(-64, 64, (n, F)) / 256.0).astype(np.float32)
    W1 = (rng.integers(-64, 64, (H, 3 + F)) / 64.0).astype(np.float32)
    # pre-activations are then odd multiples of 2^-15, never 0: no kink within a 2^-20 step
    b1 = (rng.integers(-16, 16, H) / 64.0 + 2.0 ** -15).astype(np.float32)
    W2 = (rng.integers(-64, 64, (O, H)) / 64.0).astype(np.float32)
    b2 = (rng.integers(-16, 16, O) / 64.0).astype(np.float32)
    dy = (rng.integers(-8, 8, (n, O)) / 8.0).astype(np.float32)
    return pos, x, W1, b1, W2, b2, dy


def loss(pos, x, ptr, idx, W1, b1, W2, b2, dy):
    y = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2)["y"]
    return float((y * dy.astype(np.float64)).sum())


def test_all_active_closed_form():
    """With every pre-activation positive, y_i = W2 (W1 sum_j in_ij + deg_i b1) + deg_i b2."""
    pos, x, W1, b1, W2, b2, _ = small_case(1)
    b1 = np.full_like(b1, 50.0)
    ptr, idx = relation(pos, 0.1)
    y = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2)["y"]
    n = pos.shape[0]
    for i in range(n):
        js = idx[ptr[i]:ptr[i + 1]]
        s = np.zeros(3 + x.shape[1])
        for j in js:
            s += np.concatenate([pos[j].astype(np.float64) - pos[i], x[j]])
        want = W2.astype(np.float64) @ (W1.astype(np.float64) @ s + len(js) * b1) + len(js) * b2
        np.testing.assert_allclose(y[i], want, rtol=1e-12, atol=1e-12)


def test_zero_output_layer():
    pos, x, W1, b1, W2, b2, dy = small_case(2)
    W2 = np.zeros_like(W2)
    ptr, idx = relation(pos, 0.12)
    g = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2, dy)
    deg = np.diff(ptr)
    np.testing.assert_allclose(g["y"], deg[:, None] * b2[None, :].astype(np.float64), rtol=0, atol=1e-15)
    for k in ("dx", "dp", "dW1", "db1"):
        assert np.abs(g[k]).max() == 0.0
    np.testing.assert_allclose(g["db2"], (deg[:, None] * dy).sum(0), rtol=1e-14)


def test_empty_relation():
    pos, x, W1, b1, W2, b2, dy = small_case(3)
    ptr, idx = relation(pos, 1e-6)
    assert ptr[-1] == 0
    g = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2, dy)
    for v in g.values():
        assert np.abs(v).max() == 0.0


@pytest.mark.parametrize("seed", [4, 5])
def test_gradients_by_central_differences(seed):
    pos, x, W1, b1, W2, b2, dy = small_case(seed)
    ptr, idx = relation(pos, 0.11)
    assert ptr[-1] > 20
    g = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2, dy)
    h = np.float32(2.0 ** -20)
    args = dict(pos=pos, x=x, W1=W1, b1=b1, W2=W2, b2=b2)
    want = dict(pos="dp", x="dx", W1="dW1", b1="db1", W2="dW2", b2="db2")
    rng = np.random.default_rng(seed)
    for name, gk in want.items():
        arr = args[name]
        flat = rng.choice(arr.size, size=min(arr.size, 25), replace=False)
        for f in flat:
            vals = []
            for sgn in (1, -1):
                a2 = {k: v.copy() for k, v in args.items()}
                a2[name].reshape(-1)[f] += sgn * h
                if name == "pos":   # membership is held fixed: skip a step that changes it
                    p2, i2 = relation(a2["pos"], 0.11)
                    if not (np.array_equal(p2, ptr) and np.array_equal(i2, idx)):
                        break
                vals.append(loss(a2["pos"], a2["x"], ptr, idx, a2["W1"], a2["b1"], a2["W2"], a2["b2"], dy))
            if len(vals) < 2:
                continue
            fd = (vals[0] - vals[1]) / (2 * float(h))
            an = g[gk].reshape(-1)[f]
            assert abs(fd - an) <= 1e-7 * (1 + abs(an)), (name, f, fd, an)


def test_workload_generator_shapes():
    g = synth.edgenn_inputs(n=2000, feat=8)
    assert g["pos"].shape == (2000, 3) and g["W1"].shape == (32, 11) and g["W2"].shape == (3, 32)
    ext = g["pos"].max(0) - g["pos"].min(0)
    assert abs(ext.max() - 1.0) < 1e-6


def positive_bipartite_case(seed, nd=12, ns=20, F=3, H=6, O=2, deg=7):
    """Destinations sit below every source in all three coordinates, and every feature, weight, bias
    and cotangent is positive: every displacement p_j - p_i is >= 0, every unit is active, and no
    term of any output is negative.  The relation lists `deg` random sources per destination."""
    rng = np.random.default_rng(seed)
    dst = rng.uniform(0.0, 0.4, (nd, 3))
    src = rng.uniform(0.5, 1.0, (ns, 3))
    pos = np.concatenate([dst, src]).astype(np.float32)
    n = nd + ns
    x = rng.uniform(0.1, 1.0, (n, F)).astype(np.float32)
    W1 = rng.uniform(0.1, 1.0, (H, 3 + F)).astype(np.float32)
    b1 = rng.uniform(0.1, 1.0, H).astype(np.float32)
    W2 = rng.uniform(0.1, 1.0, (O, H)).astype(np.float32)
    b2 = rng.uniform(0.1, 1.0, O).astype(np.float32)
    dy = rng.uniform(0.1, 1.0, (n, O)).astype(np.float32)
    lists = [np.sort(rng.choice(ns, deg, replace=False)) + nd for _ in range(nd)] + [np.array([], int)] * ns
    ptr = np.zeros(n + 1, np.int64)
    ptr[1:] = np.cumsum([len(l) for l in lists])
    idx = np.concatenate(lists).astype(np.int32)
    return pos, x, W1, b1, W2, b2, dy, ptr, idx, nd


@pytest.mark.parametrize("seed", [11, 12])
def test_magnitudes_equal_values_when_every_term_is_positive(seed):
    """With no negative term anywhere, each output's absolute-value evaluation is the output itself
    (destinations' position gradients are minus a positive sum).  A dropped or misplaced term in any
    of the seven magnitudes breaks an equality here."""
    pos, x, W1, b1, W2, b2, dy, ptr, idx, nd = positive_bipartite_case(seed)
    val, mag, slack = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2, dy, terms=True)
    for k in ("y", "dx", "dW1", "db1", "dW2", "db2"):
        assert np.array_equal(mag[k], val[k]), k
        assert val[k].max() > 0, k
    assert np.array_equal(mag["dp"][nd:], val["dp"][nd:])     # sources: + sum of positive terms
    assert np.array_equal(mag["dp"][:nd], -val["dp"][:nd])    # destinations: - the same kind of sum
    assert np.all(val["dp"][:nd] < 0) and np.all(val["dp"][nd:] >= 0)
    for k, s in slack.items():
        assert not s.any(), k


def test_slack_bounds_the_jump_of_an_unsettled_relu():
    """A unit whose pre-activation is exactly 0 at one pair has an unsettled decision.  Moving b1 of
    that unit by one fp32 unit up or down flips the decision; every gradient output changes by at
    most its slack (plus the first-order change), and the outputs with no slack do not jump."""
    pos, x, W1, b1, W2, b2, dy = small_case(21)
    ptr, idx = relation(pos, 0.11)
    i0 = int(np.argmax(np.diff(ptr)))
    j0 = int(idx[ptr[i0]])
    h = 2
    inp = np.concatenate([pos[j0].astype(np.float64) - pos[i0], x[j0].astype(np.float64)])
    b1 = b1.copy()
    b1[h] = np.float32(-(W1[h].astype(np.float64) @ inp))   # exact: every product is a multiple of 2^-14
    assert float(b1[h]) == -(W1[h].astype(np.float64) @ inp)
    val, mag, slack = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2, dy, terms=True)
    assert slack["db1"][h] > 0 and slack["dx"][j0].max() > 0
    step = np.float32(2.0 ** -20)   # |b1| < 2: exact steps; every other pre-activation is >= 2^-14 away
    outs = []
    for sgn in (1, -1):
        b = b1.copy()
        b[h] = b[h] + sgn * step
        outs.append(oracle.edgenn(pos, x, ptr, idx, W1, b, W2, b2, dy))
    jumped = False
    for k in ("dx", "dp", "dW1", "db1", "dW2"):
        jump = np.abs(outs[0][k] - outs[1][k])
        first_order = 1e-5 * (mag[k] + slack[k]) + 1e-12
        assert np.all(jump <= slack[k] + first_order), k
        assert np.all(jump[slack[k] == 0] <= first_order[slack[k] == 0]), k
        jumped |= bool((jump > first_order).any())
    assert jumped
    # a pre-activation 2^-20 from zero, far below 2^-14 of its magnitude, is still unsettled
    aa = float(np.abs(W1[h]).astype(np.float64) @ np.abs(inp)) + abs(float(b1[h]))
    assert 2.0 ** -20 < 2.0 ** -14 * aa
    b = b1.copy()
    b[h] = b[h] + np.float32(2.0 ** -20)
    assert oracle.edgenn(pos, x, ptr, idx, W1, b, W2, b2, dy, terms=True)[2]["db1"][h] > 0


def test_magnitudes_bound_values_on_mixed_signs():
    pos, x, W1, b1, W2, b2, dy = small_case(22)
    ptr, idx = relation(pos, 0.12)
    val, mag, _ = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2, dy, terms=True)
    for k in val:
        assert np.all(np.abs(val[k]) <= mag[k] * (1 + 1e-15)), k
        assert (mag[k] > np.abs(val[k])).any(), k     # cancellation happens: not a copy of |value|


def test_magnitudes_of_one_pair_closed_form():
    """One destination with one source and mixed signs everywhere, written out from the definition
    (numpy, vectorized): the pre-activation magnitudes aa = |b1| + |W1| |in|, the active set of the
    true pre-activations, y's magnitude |b2| + |W2| (active * aa), the cotangent magnitudes
    g = |W2|^T |dy| and the input-gradient magnitudes |W1|^T (active * g)."""
    rng = np.random.default_rng(23)
    F, H, O = 2, 7, 3
    pos = np.array([[0.25, -0.5, 0.125], [-0.375, 0.25, 0.5]], np.float32)
    x = rng.uniform(-1, 1, (2, F)).astype(np.float32)
    W1 = rng.uniform(-1, 1, (H, 3 + F)).astype(np.float32)
    b1 = rng.uniform(-0.5, 0.5, H).astype(np.float32)
    W2 = rng.uniform(-1, 1, (O, H)).astype(np.float32)
    b2 = rng.uniform(-1, 1, O).astype(np.float32)
    dy = rng.uniform(-1, 1, (2, O)).astype(np.float32)
    ptr = np.array([0, 1, 1], np.int64)
    idx = np.array([1], np.int32)
    val, mag, slack = oracle.edgenn(pos, x, ptr, idx, W1, b1, W2, b2, dy, terms=True)
    inp = np.concatenate([pos[1].astype(np.float64) - pos[0], x[1]])
    a = W1.astype(np.float64) @ inp + b1
    act = a > 0
    assert 0 < act.sum() < H
    aa = np.abs(W1).astype(np.float64) @ np.abs(inp) + np.abs(b1)
    g = np.abs(W2).astype(np.float64).T @ np.abs(dy[0]).astype(np.float64)
    np.testing.assert_allclose(mag["y"][0], np.abs(b2) + np.abs(W2) @ (act * aa), rtol=1e-14)
    assert not mag["y"][1].any()
    din = np.abs(W1).astype(np.float64).T @ (act * g)
    np.testing.assert_allclose(mag["dx"][1], din[3:], rtol=1e-14)
    np.testing.assert_allclose(mag["dp"][0], din[:3], rtol=1e-14)
    np.testing.assert_allclose(mag["dp"][1], din[:3], rtol=1e-14)
    np.testing.assert_allclose(mag["dW1"], np.outer(act * g, np.abs(inp)), rtol=1e-14)
    np.testing.assert_allclose(mag["db1"], act * g, rtol=1e-14)
    np.testing.assert_allclose(mag["dW2"], np.outer(np.abs(dy[0]), act * aa), rtol=1e-14)
    np.testing.assert_allclose(mag["db2"], np.abs(dy[0]), rtol=1e-14)
    for s in slack.values():
        assert not s.any()
