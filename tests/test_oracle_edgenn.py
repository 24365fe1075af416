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
