"""The CSR forward and gather-mode backward inside a captured HIP graph.

Both paths clear memory with fill kernels (no hipMemsetAsync) and never synchronize, so a caller
can capture a launch-bound step (config 1: 1,024 nodes, 8,192 edges) once and replay it.  Every
replay, with new inputs copied into the captured buffers and eager calls in between, must give the
eager result bit for bit (the kernels are deterministic)."""
import numpy as np
import pytest
import torch

from paper_2609_24802_amd import synth

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("reducer", ["sum", "max"])
def test_forward_backward_replayed_in_a_graph(lib, reducer):
    g = synth.csr_uniform_small()
    red = lib.REDUCE_SUM if reducer == "sum" else lib.REDUCE_MAX
    rel = lib.Csr(dev(g["row_ptr"]), dev(g["col"]), g["num_src"])
    rev = lib.tiga_csr_transpose(rel)
    rng = np.random.default_rng(8)
    xs = [dev(rng.uniform(-1, 1, g["x"].shape).astype(np.float32)) for _ in range(3)]
    dys = [dev(rng.standard_normal(g["dy"].shape).astype(np.float32)) for _ in range(3)]
    w = dev(g["w"])
    x_in, dy_in = xs[0].clone(), dys[0].clone()

    def step(x, dy):
        y, arg = lib.tiga_mp_csr_fwd(rel, x, w, reducer=red)
        dx, dw = lib.tiga_mp_csr_bwd(rel, dy, x, w, reducer=red, argmax=arg, rev=rev)
        return y, arg, dx, dw

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):
            step(x_in, dy_in)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        out = step(x_in, dy_in)
    for i in range(4):
        x_in.copy_(xs[i % 3])
        dy_in.copy_(dys[(i + 1) % 3])
        graph.replay()
        ref = step(xs[i % 3], dys[(i + 1) % 3])     # eager work between the replays
        torch.cuda.synchronize()
        for got, want in zip(out, ref):
            if want is None:
                assert got is None
            else:
                assert torch.equal(got, want), (reducer, i)
