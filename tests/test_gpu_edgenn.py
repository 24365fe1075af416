"""GPU parity of the edge-local MLP message (forward and every gradient) against the oracle.

The oracle runs the same message and VJP in fp64 over the oracle's own radius relation and returns,
for every output, its absolute-value evaluation (the sum|terms| of a composed expression) and the
slack of ReLU decisions that fp32 cannot settle.  Every output must satisfy
|gpu - oracle| <= 1e-5 * sum|terms| + slack, and an output with no terms must be exactly 0."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_24802_amd import synth
from tests.parity import assert_terms_close

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def case(n, F, H, O, radius, seed, surface=False):
    pos = synth.surface_points(n, (70, n, seed)) if surface else synth.uniform_f32(n * 3, 0, 1, (71, n, seed)).reshape(n, 3)
    x = synth.normal_f32(max(n * F, 1), (72, n, F, seed))[: n * F].reshape(n, F)
    prm = synth.mlp_params(3 + F, H, O, (73, F, H, O, seed))
    dy = synth.normal_f32(n * O, (74, n, O, seed)).reshape(n, O)
    return pos, x, np.float32(radius), prm, dy


def check(lib, pos, x, radius, prm, dy):
    n, F = x.shape
    ptr, idx = oracle.radius_neighbors(pos, radius)
    ref, mag, slack = oracle.edgenn(pos, x, ptr, idx, prm["W1"], prm["b1"], prm["W2"], prm["b2"], dy, terms=True)
    args = (dev(pos), dev(x) if F else None, radius, dev(prm["W1"]), dev(prm["b1"]), dev(prm["W2"]), dev(prm["b2"]))
    y = lib.tiga_mp_edgenn_fwd(*args)
    g = lib.tiga_mp_edgenn_bwd(*args, dev(dy))
    torch.cuda.synchronize()
    assert_terms_close(y.cpu().numpy(), ref["y"], mag["y"], what="y", slack=slack["y"])
    for k, rk in (("dpos", "dp"), ("dW1", "dW1"), ("db1", "db1"), ("dW2", "dW2"), ("db2", "db2")) + \
            ((("dx", "dx"),) if F else ()):
        assert_terms_close(g[k].cpu().numpy(), ref[rk], mag[rk], what=k, slack=slack[rk])
    return int(ptr[-1])


@pytest.mark.parametrize("n,F,H,O,r", [(300, 8, 16, 4, 0.15), (500, 0, 32, 3, 0.12), (400, 3, 5, 1, 0.13),
                                       (600, 32, 32, 3, 0.1), (256, 64, 64, 8, 0.2), (350, 16, 64, 2, 0.14),
                                       (1, 8, 32, 3, 0.1), (2000, 8, 32, 3, 0.06), (900, 12, 20, 5, 0.09),
                                       (700, 24, 12, 2, 0.11)])
def test_edgenn_against_oracle(lib, n, F, H, O, r):
    check(lib, *case(n, F, H, O, r, seed=n + F + H))


def test_edgenn_empty_relation(lib):
    pos, x, _, prm, dy = case(200, 8, 16, 3, 0.1, seed=9)
    edges = check(lib, pos, x, np.float32(1e-6), prm, dy)
    assert edges == 0


@pytest.mark.parametrize("F", [8, 32])
def test_edgenn_surface_workload(lib, F):
    """The measured workload: 35,947 surface points, radius 0.015, hidden 32, 3 outputs."""
    g = synth.edgenn_inputs(feat=F)
    prm = {k: g[k] for k in ("W1", "b1", "W2", "b2")}
    edges = check(lib, g["pos"], g["x"], g["radius"], prm, g["dy"])
    assert edges > 200_000


def test_edgenn_autograd_wrapper(lib):
    pos, x, r, prm, dy = case(400, 8, 16, 3, 0.15, seed=3)
    t = [dev(a).requires_grad_() for a in (pos, x, prm["W1"], prm["b1"], prm["W2"], prm["b2"])]
    y = lib.edge_mlp(*t, float(r))
    y.backward(dev(dy))
    direct = lib.tiga_mp_edgenn_bwd(*[a.detach() for a in t[:2]], float(r), *[a.detach() for a in t[2:]], dev(dy))
    for a, k in zip(t, ("dpos", "dx", "dW1", "db1", "dW2", "db2")):
        assert torch.equal(a.grad, direct[k]), k
