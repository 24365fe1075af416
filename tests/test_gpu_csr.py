"""GPU parity of the CSR entry points against the oracle.

Floating-point sums: |gpu - oracle| <= 1e-5 * sum|terms| per output.
Integer-valued inputs make every fp32 partial sum exact, so those cases are
compared bit for bit.  Max values and argmax are always bit-exact.
"""
import json
import re
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_24802_amd import synth
from tests.parity import assert_terms_close

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.cpu().numpy()


def make_graph(degrees, num_src, F, seed, integer=False):
    """CSR with the given row degrees, uniform sources (duplicates/self loops arise naturally)."""
    rng = np.random.default_rng(seed)
    deg = np.asarray(degrees, np.int64)
    row_ptr = np.zeros(deg.size + 1, np.int64)
    np.cumsum(deg, out=row_ptr[1:])
    E = int(row_ptr[-1])
    col = rng.integers(0, num_src, E).astype(np.int32)
    if integer:
        x = rng.integers(-3, 4, (num_src, F)).astype(np.float32)
        w = rng.integers(0, 3, E).astype(np.float32)
        dy = rng.integers(-2, 3, (deg.size, F)).astype(np.float32)
    else:
        x = rng.standard_normal((num_src, F)).astype(np.float32)
        w = rng.random(E).astype(np.float32)
        dy = rng.standard_normal((deg.size, F)).astype(np.float32)
    return row_ptr, col, x, w, dy


def mixed_degrees(n, seed, big=()):
    """Short, medium and long rows in random order, plus empty rows and the given huge rows."""
    rng = np.random.default_rng(seed)
    d = rng.choice([0, 1, 2, 3, 5, 8, 9, 16, 17, 31, 64, 100, 257, 700, 1100, 2500, 5000], size=n,
                   p=[.08, .1, .1, .1, .1, .1, .05, .05, .05, .05, .05, .04, .04, .03, .02, .02, .02])
    for k, b in enumerate(big):
        d[(k * 7919) % n] = b
    return d


def run_fwd(lib, row_ptr, col, x, w, num_src, reducer):
    rel = lib.Csr(dev(row_ptr), dev(col), num_src)
    y, arg = lib.tiga_mp_csr_fwd(rel, dev(x), dev(w) if w is not None else None, reducer=reducer)
    torch.cuda.synchronize()
    return rel, host(y), (host(arg) if arg is not None else None)


def test_worked_example(lib):
    g = json.load(open(GOLD))
    rp, col = np.array(g["row_ptr"], np.int64), np.array(g["col_idx"], np.int32)
    x = np.array(g["x"], np.float32)[:, None]
    w = np.array(g["w"], np.float32)
    dy = np.array(g["dy"], np.float32)[:, None]
    rel, y, _ = run_fwd(lib, rp, col, x, w, g["num_src"], lib.REDUCE_SUM)
    assert y[:, 0].tolist() == g["printed"]["y"]
    rev = lib.tiga_csr_transpose(rel)
    for r in (None, rev):
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), rev=r)
        assert host(dx)[:, 0].tolist() == g["printed"]["dx"]
        assert host(dw).tolist() == g["printed"]["dw"]
    rel, y, arg = run_fwd(lib, rp, col, x, w, g["num_src"], lib.REDUCE_MAX)
    d = g["derived_max"]
    assert y[:, 0].tolist() == d["y"] and arg[:, 0].tolist() == d["arg"]
    for r in (None, rev):
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), reducer=lib.REDUCE_MAX, argmax=dev(arg), rev=r)
        assert host(dx)[:, 0].tolist() == d["dx"] and host(dw).tolist() == d["dw"]


@pytest.mark.parametrize("F", [1, 3, 16, 17, 32, 64, 128, 260])
def test_sum_forward_mixed_degrees(lib, F):
    deg = mixed_degrees(900, F, big=(20000,) if F <= 64 else ())
    row_ptr, col, x, w, dy = make_graph(deg, 700, F, seed=F)
    _, y, _ = run_fwd(lib, row_ptr, col, x, w, 700, lib.REDUCE_SUM)
    ref, mag = oracle.csr_sum_fwd(row_ptr, col, x, w)
    assert_terms_close(y, ref, mag, what=f"sum F={F}")
    # unweighted message
    _, y1, _ = run_fwd(lib, row_ptr, col, x, None, 700, lib.REDUCE_SUM)
    ref1, mag1 = oracle.csr_sum_fwd(row_ptr, col, x, None)
    assert_terms_close(y1, ref1, mag1, what=f"sum unweighted F={F}")


@pytest.mark.parametrize("F", [1, 4, 16, 17, 64])
def test_sum_integer_inputs_bit_exact(lib, F):
    deg = mixed_degrees(1200, 100 + F, big=(30000, 4097))
    row_ptr, col, x, w, dy = make_graph(deg, 1500, F, seed=F + 7, integer=True)
    rel, y, _ = run_fwd(lib, row_ptr, col, x, w, 1500, lib.REDUCE_SUM)
    ref, _ = oracle.csr_sum_fwd(row_ptr, col, x, w)
    assert np.array_equal(y, ref.astype(np.float32))
    rdx, _, rdw, _ = oracle.csr_sum_bwd(row_ptr, col, x, w, dy, 1500)
    rev = lib.tiga_csr_transpose(rel)
    for r in (None, rev):
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), rev=r)
        assert np.array_equal(host(dx), rdx.astype(np.float32))
        assert np.array_equal(host(dw), rdw.astype(np.float32))


@pytest.mark.parametrize("F", [1, 3, 16, 17, 64, 260])
def test_max_forward_backward_exact(lib, F):
    deg = mixed_degrees(800, 200 + F, big=(12000,))
    row_ptr, col, x, w, dy = make_graph(deg, 600, F, seed=F + 11)
    rel, y, arg = run_fwd(lib, row_ptr, col, x, w, 600, lib.REDUCE_MAX)
    ry, rarg = oracle.csr_max_fwd(row_ptr, col, x, w)
    assert np.array_equal(arg, rarg)
    assert np.array_equal(y.view(np.int32), ry.view(np.int32))  # bit patterns, -0 included
    rdx, rdxa, rdw, rdwa = oracle.csr_max_bwd(row_ptr, col, x, w, rarg, dy, 600)
    rev = lib.tiga_csr_transpose(rel)
    for r in (None, rev):
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), reducer=lib.REDUCE_MAX, argmax=dev(arg), rev=r)
        assert_terms_close(host(dx), rdx, rdxa, what=f"max dx F={F} rev={r is not None}")
        assert_terms_close(host(dw), rdw, rdwa, what=f"max dw F={F}")


@pytest.mark.parametrize("F", [12, 20, 44, 260])
def test_atomic_backward_ragged_unit_blocks(lib, F):
    """Atomic-mode dx at widths whose last block of 16-byte units is partly outside the row: the
    lane-contiguous scatter must cover exactly the row's F floats. Integer inputs make every sum
    exact, so the order of the atomics does not matter."""
    deg = mixed_degrees(700, 300 + F, big=(9000,))
    row_ptr, col, x, w, dy = make_graph(deg, 900, F, seed=F + 31, integer=True)
    rel, _, _ = run_fwd(lib, row_ptr, col, x, w, 900, lib.REDUCE_SUM)
    rdx, _, rdw, _ = oracle.csr_sum_bwd(row_ptr, col, x, w, dy, 900)
    dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w))
    assert np.array_equal(host(dx), rdx.astype(np.float32))
    assert np.array_equal(host(dw), rdw.astype(np.float32))
    _, _, arg = run_fwd(lib, row_ptr, col, x, w, 900, lib.REDUCE_MAX)
    _, rarg = oracle.csr_max_fwd(row_ptr, col, x, w)
    assert np.array_equal(arg, rarg)
    mdx, _, mdw, _ = oracle.csr_max_bwd(row_ptr, col, x, w, rarg, dy, 900)
    dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), reducer=lib.REDUCE_MAX, argmax=dev(arg))
    assert np.array_equal(host(dx), mdx.astype(np.float32))
    assert np.array_equal(host(dw), mdw.astype(np.float32))


@pytest.mark.parametrize("num_src,hot", [(3_000_000, 40), (200, 0), (70_000, 5)])
def test_transpose_is_a_stable_sort_by_source(lib, num_src, hot):
    """The reverse incidence lists each source's edges in forward-edge order: numpy's stable
    argsort of col fixes edge_id and src_ptr exactly (1 to 3 radix passes, many tiles,
    a ragged last tile, and hot sources whose runs span tiles)."""
    rng = np.random.default_rng(num_src + hot)
    deg = rng.integers(0, 9, 40_000)
    deg[rng.integers(0, deg.size, 30)] = 3000
    rp = np.zeros(deg.size + 1, np.int64)
    np.cumsum(deg, out=rp[1:])
    e = int(rp[-1])
    col = rng.integers(0, num_src, e).astype(np.int32)
    if hot:
        pick = rng.random(e) < 0.3
        col[pick] = rng.integers(0, hot, int(pick.sum()))
    rev = lib.tiga_csr_transpose(lib.Csr(dev(rp), dev(col), num_src))
    torch.cuda.synchronize()
    order = np.argsort(col, kind="stable")
    ptr = np.zeros(num_src + 1, np.int64)
    np.cumsum(np.bincount(col, minlength=num_src), out=ptr[1:])
    assert np.array_equal(host(rev.edge_id), order.astype(np.int32))
    assert np.array_equal(host(rev.src_ptr), ptr)


def test_max_ties_and_signed_zeros(lib):
    # duplicated edges with equal weights, all-zero rows of x, and w = 0 with
    # negative x (a -0 message) next to +0 messages
    F = 8
    deg = mixed_degrees(500, 5, big=(9000,))
    row_ptr, col, x, w, dy = make_graph(deg, 40, F, seed=5)
    x[::3] = 0.0
    w[::5] = 0.0
    x = np.round(x)  # many equal messages
    w = np.round(w * 2) / 2
    rel, y, arg = run_fwd(lib, row_ptr, col, x, w, 40, lib.REDUCE_MAX)
    ry, rarg = oracle.csr_max_fwd(row_ptr, col, x, w)
    assert np.array_equal(arg, rarg)
    assert np.array_equal(y.view(np.int32), ry.view(np.int32))


def test_sum_backward_random(lib):
    F = 32
    deg = mixed_degrees(1000, 9, big=(40000,))
    row_ptr, col, x, w, dy = make_graph(deg, 1300, F, seed=9)
    rel = lib.Csr(dev(row_ptr), dev(col), 1300)
    rdx, rdxa, rdw, rdwa = oracle.csr_sum_bwd(row_ptr, col, x, w, dy, 1300)
    rev = lib.tiga_csr_transpose(rel)
    outs = []
    for r in (None, rev, rev):
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), rev=r)
        assert_terms_close(host(dx), rdx, rdxa, what="sum dx")
        assert_terms_close(host(dw), rdw, rdwa, what="sum dw")
        outs.append((host(dx), host(dw)))
    # the reverse-incidence gather is deterministic
    assert np.array_equal(outs[1][0], outs[2][0]) and np.array_equal(outs[1][1], outs[2][1])


@pytest.mark.parametrize("F", [1, 3, 16, 17, 64, 260])
def test_sum_backward_gather_modes(lib, F):
    """With the reverse incidence: both gradients in one traversal (rows of one
    feature block), dw from the edge kernel when the row needs several blocks,
    and each gradient alone."""
    deg = mixed_degrees(600, 21 + F, big=(9000,))
    row_ptr, col, x, w, dy = make_graph(deg, 700, F, seed=21 + F)
    rel = lib.Csr(dev(row_ptr), dev(col), 700)
    rdx, rdxa, rdw, rdwa = oracle.csr_sum_bwd(row_ptr, col, x, w, dy, 700)
    rev = lib.tiga_csr_transpose(rel)
    dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), rev=rev)
    assert_terms_close(host(dx), rdx, rdxa, what=f"sum dx F={F}")
    assert_terms_close(host(dw), rdw, rdwa, what=f"sum dw F={F}")
    dx1, none = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), rev=rev, want_dw=False)
    assert none is None
    assert_terms_close(host(dx1), rdx, rdxa, what=f"sum dx alone F={F}")
    none, dw1 = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), rev=rev, want_dx=False)
    assert none is None
    assert_terms_close(host(dw1), rdw, rdwa, what=f"sum dw alone F={F}")


def test_kernel_events_last_one_call(lib):
    """Events armed before a call without a fused kernel (the transpose) are
    dropped by it: the next forward records nothing into them."""
    deg = mixed_degrees(300, 5)
    row_ptr, col, x, w, _ = make_graph(deg, 400, 16, seed=5)
    rel = lib.Csr(dev(row_ptr), dev(col), 400)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    b.record()
    torch.cuda.synchronize()
    before = a.elapsed_time(b)
    lib.tiga_mp_set_kernel_events(a, b)
    lib.tiga_csr_transpose(rel)
    lib.tiga_mp_csr_fwd(rel, dev(x), dev(w))
    torch.cuda.synchronize()
    assert a.elapsed_time(b) == before
    # armed right before a forward, the events bracket its kernel
    lib.tiga_mp_set_kernel_events(a, b)
    lib.tiga_mp_csr_fwd(rel, dev(x), dev(w))
    torch.cuda.synchronize()
    assert a.elapsed_time(b) != before


def test_transpose_is_stable_sort(lib):
    deg = mixed_degrees(3000, 13, big=(70000,))
    row_ptr, col, *_ = make_graph(deg, 100_000, 1, seed=13)
    col[:5000] = 77  # a hub source
    rel = lib.Csr(dev(row_ptr), dev(col), 100_000)
    rev = lib.tiga_csr_transpose(rel)
    order = np.argsort(col, kind="stable")
    assert np.array_equal(host(rev.edge_id), order)
    sp = np.zeros(100_001, np.int64)
    np.cumsum(np.bincount(col, minlength=100_000), out=sp[1:])
    assert np.array_equal(host(rev.src_ptr), sp)


def test_empty_and_degenerate(lib):
    # no edges at all; a single row; rectangular with num_src > num_dst
    for degs, ns in [([0, 0, 0], 4), ([5], 1), ([0, 3, 0, 2], 9)]:
        row_ptr, col, x, w, dy = make_graph(degs, ns, 4, seed=1)
        rel, y, _ = run_fwd(lib, row_ptr, col, x, w, ns, lib.REDUCE_SUM)
        ref, mag = oracle.csr_sum_fwd(row_ptr, col, x, w)
        assert_terms_close(y, ref, mag)
        rel, ym, am = run_fwd(lib, row_ptr, col, x, w, ns, lib.REDUCE_MAX)
        rym, ram = oracle.csr_max_fwd(row_ptr, col, x, w)
        assert np.array_equal(am, ram) and np.array_equal(ym, rym)
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w))
        rdx, _, rdw, _ = oracle.csr_sum_bwd(row_ptr, col, x, w, dy, ns)
        assert np.allclose(host(dx), rdx) and np.allclose(host(dw), rdw)


def test_validation(lib):
    row_ptr = np.array([0, 2, 3, 3], np.int64)
    col = np.array([0, 1, 1], np.int32)
    lib.tiga_csr_validate(lib.Csr(dev(row_ptr), dev(col), 2))
    bad = [
        (np.array([1, 2, 3, 3]), col, 2, "row_ptr[0]"),
        (np.array([0, 3, 2, 3]), col, 2, "decreases"),
        (row_ptr, np.array([0, 2, 1], np.int32), 2, "col_idx[1]"),
        (row_ptr, np.array([0, -1, 1], np.int32), 2, "col_idx[1]"),
    ]
    for rp, c, ns, msg in bad:
        with pytest.raises(lib.TigaError, match=re.escape(msg)) as e:
            lib.tiga_csr_validate(lib.Csr(dev(rp.astype(np.int64)), dev(c.astype(np.int32)), ns))
        assert e.value.code == lib.TIGA_EGRAPH


def test_config1_uniform_small(lib):
    g = synth.csr_uniform_small()
    rp, col, x, w, dy = g["row_ptr"], g["col"], g["x"], g["w"], g["dy"]
    rel, y, _ = run_fwd(lib, rp, col, x, w, 1024, lib.REDUCE_SUM)
    ref, mag = oracle.csr_sum_fwd(rp, col, x, w)
    assert_terms_close(y, ref, mag, what="config 1 y")
    rdx, rdxa, rdw, rdwa = oracle.csr_sum_bwd(rp, col, x, w, dy, 1024)
    rev = lib.tiga_csr_transpose(rel)
    for r in (None, rev):
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), rev=r)
        assert_terms_close(host(dx), rdx, rdxa, what="config 1 dx")
        assert_terms_close(host(dw), rdw, rdwa, what="config 1 dw")


def _sample_rows(row_ptr, k, seed):
    deg = np.diff(row_ptr)
    rng = np.random.default_rng(seed)
    top = np.argsort(-deg, kind="stable")[:8]  # the split rows
    return np.unique(np.concatenate([top, rng.integers(0, deg.size, k), [0, deg.size - 1]]))


def test_config2_powerlaw_full_size(lib):
    g = synth.config2()
    rp, col, x, w, dy, n = g["row_ptr"], g["col"], g["x"], g["w"], g["dy"], g["num_dst"]
    rel = lib.Csr(dev(rp), dev(col), n)
    xd, wd, dyd = dev(x), dev(w), dev(dy)
    rows = _sample_rows(rp, 3000, 2)
    y, _ = lib.tiga_mp_csr_fwd(rel, xd, wd)
    ref, mag = oracle.csr_sum_fwd(rp, col, x, w, rows=rows)
    assert_terms_close(host(y)[rows], ref, mag, what="config 2 sum y")
    ym, am = lib.tiga_mp_csr_fwd(rel, xd, wd, reducer=lib.REDUCE_MAX)
    rym, ram = oracle.csr_max_fwd(rp, col, x, w, rows=rows)
    assert np.array_equal(host(am)[rows], ram) and np.array_equal(host(ym)[rows], rym)
    # full-size backward: every dw of the sampled rows' edges and sampled dx rows
    rdx, rdxa, rdw, rdwa = oracle.csr_sum_bwd(rp, col, x, w, dy, n)
    rev = lib.tiga_csr_transpose(rel)
    src = np.random.default_rng(3).integers(0, n, 3000)
    edges = np.concatenate([np.arange(rp[r], rp[r + 1]) for r in rows])
    for r in (None, rev):
        dx, dw = lib.tiga_mp_csr_bwd(rel, dyd, xd, wd, rev=r)
        assert_terms_close(host(dx)[src], rdx[src], rdxa[src], what="config 2 sum dx")
        assert_terms_close(host(dw)[edges], rdw[edges], rdwa[edges], what="config 2 sum dw")
    am_h = host(am)
    rdx, rdxa, rdw, rdwa = oracle.csr_max_bwd(rp, col, x, w, am_h, dy, n)
    for r in (None, rev):
        dx, dw = lib.tiga_mp_csr_bwd(rel, dyd, xd, wd, reducer=lib.REDUCE_MAX, argmax=am, rev=r)
        assert_terms_close(host(dx)[src], rdx[src], rdxa[src], what="config 2 max dx")
        assert_terms_close(host(dw)[edges], rdw[edges], rdwa[edges], what="config 2 max dw")


@pytest.mark.slow
def test_config5_billion_edges_full(lib):
    """Every one of the 50M output rows of the 1e9-edge graph against the oracle (in row blocks, so
    the fp64 references stay a few GB; the oracle takes a few seconds of the host's cores)."""
    g = synth.config5()
    rp, col, x, w, n = g["row_ptr"], g["col"], g["x"], g["w"], g["num_dst"]
    rel = lib.Csr(dev(rp), dev(col), n)
    xd, wd = dev(x), dev(w)
    y, _ = lib.tiga_mp_csr_fwd(rel, xd, wd)
    yh = host(y)
    block = 5_000_000
    for a in range(0, n, block):
        rows = np.arange(a, min(n, a + block), dtype=np.int64)
        ref, mag = oracle.csr_sum_fwd(rp, col, x, w, rows=rows)
        assert_terms_close(yh[a:a + rows.size], ref, mag, what=f"config 5 y rows {a}..")
        print(f"config 5: rows {a + rows.size} of {n} checked", flush=True)
        del ref, mag
    # the column sums of y equal the out-weight-scaled column sums of x (all rows)
    outw = torch.zeros(n, dtype=torch.float64, device="cuda")
    outw.index_add_(0, rel.col_idx.long(), wd.double())
    lhs = y.double().sum(0)
    rhs = (outw[:, None] * xd.double()).sum(0)
    scale = (outw[:, None] * xd.double().abs()).sum(0)
    assert torch.all((lhs - rhs).abs() <= 1e-5 * scale)


@pytest.mark.parametrize("reducer,use_rev", [(0, False), (0, True), (1, True)])
def test_autograd_wrapper(lib, reducer, use_rev):
    """csr_aggregate's backward returns exactly the direct VJP call's gradients."""
    F = 16
    deg = mixed_degrees(500, 31)
    row_ptr, col, x, w, dy = make_graph(deg, 450, F, seed=31)
    rel = lib.Csr(dev(row_ptr), dev(col), 450)
    rev = lib.tiga_csr_transpose(rel) if use_rev else None
    xt = dev(x).requires_grad_(True)
    wt = dev(w).requires_grad_(True)
    y, arg = lib.csr_aggregate(rel, xt, wt, reducer=reducer, rev=rev)
    y.backward(dev(dy))
    ref_y, ref_arg = lib.tiga_mp_csr_fwd(rel, dev(x), dev(w), reducer=reducer)
    assert torch.equal(y.detach(), ref_y)
    dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), reducer=reducer, argmax=ref_arg, rev=rev)
    if use_rev:  # deterministic: identical bits
        assert torch.equal(xt.grad, dx) and torch.equal(wt.grad, dw)
    rdx, rdxa, rdw, rdwa = (oracle.csr_sum_bwd(row_ptr, col, x, w, dy, 450) if reducer == 0 else
                            oracle.csr_max_bwd(row_ptr, col, x, w, host(ref_arg), dy, 450))
    assert_terms_close(host(xt.grad), rdx, rdxa, what="autograd dx")
    assert_terms_close(host(wt.grad), rdw, rdwa, what="autograd dw")


def test_sum_forward_all_positive_long_rows(lib):
    """All-positive messages make sum|terms| equal |y|, so the 1e-5 bound is a
    true relative-error bound; rows of 2e5 and 1e6 edges are split into many
    chunks and merged."""
    F = 16
    deg = mixed_degrees(400, 51, big=(200_000, 1_000_000))
    row_ptr, col, _, _, _ = make_graph(deg, 50_000, F, seed=51)
    rng = np.random.default_rng(52)
    x = rng.random((50_000, F)).astype(np.float32) + np.float32(0.5)
    w = rng.random(col.size).astype(np.float32) + np.float32(0.5)
    rel, y, _ = run_fwd(lib, row_ptr, col, x, w, 50_000, lib.REDUCE_SUM)
    ry, rya = oracle.csr_sum_fwd(row_ptr, col, x, w)
    assert np.allclose(rya, np.abs(ry))
    assert_terms_close(y, ry, rya, what="all-positive sum")


def test_forward_bit_identical_across_runs(lib):
    """Sum and max forwards are deterministic: split rows merge in a fixed order."""
    F = 32
    deg = mixed_degrees(2000, 53, big=(150_000, 40_000))
    row_ptr, col, x, w, _ = make_graph(deg, 3000, F, seed=53)
    rel = lib.Csr(dev(row_ptr), dev(col), 3000)
    xd, wd = dev(x), dev(w)
    for red in (lib.REDUCE_SUM, lib.REDUCE_MAX):
        a, aa = lib.tiga_mp_csr_fwd(rel, xd, wd, reducer=red)
        b, bb = lib.tiga_mp_csr_fwd(rel, xd, wd, reducer=red)
        assert torch.equal(a, b)
        if red == lib.REDUCE_MAX:
            assert torch.equal(aa, bb)


@pytest.mark.parametrize("num_edges", [1 << 16, (1 << 16) + 1])
@pytest.mark.parametrize("reducer", ["sum", "max"])
def test_direct_traversal_boundary(lib, num_edges, reducer):
    """Relations of at most 2^16 edges (and rows) take the single-launch traversal, larger ones the
    planned one.  Both sides of the boundary, each with a row of about 60,000 edges and empty rows:
    forward and gather-mode backward against the oracle."""
    n, F = 500, 16
    rng = np.random.default_rng(num_edges)
    deg = rng.integers(0, 23, n).astype(np.int64)
    deg[100] = 0
    deg[100] = num_edges - int(deg.sum())
    assert deg[100] > 50000 and (deg == 0).any()
    row_ptr, col, x, w, dy = make_graph(deg, 400, F, seed=int(num_edges % 97))
    red = lib.REDUCE_SUM if reducer == "sum" else lib.REDUCE_MAX
    rel, y, arg = run_fwd(lib, row_ptr, col, x, w, 400, red)
    rev = lib.tiga_csr_transpose(rel)
    if reducer == "sum":
        ry, rya = oracle.csr_sum_fwd(row_ptr, col, x, w)
        assert_terms_close(y, ry, rya, what=f"direct boundary sum E={num_edges}")
        rdx, rdxa, rdw, rdwa = oracle.csr_sum_bwd(row_ptr, col, x, w, dy, 400)
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), rev=rev)
    else:
        ry, rarg = oracle.csr_max_fwd(row_ptr, col, x, w)
        assert np.array_equal(arg, rarg)
        assert np.array_equal(y.view(np.int32), ry.view(np.int32))
        rdx, rdxa, rdw, rdwa = oracle.csr_max_bwd(row_ptr, col, x, w, rarg, dy, 400)
        dx, dw = lib.tiga_mp_csr_bwd(rel, dev(dy), dev(x), dev(w), reducer=lib.REDUCE_MAX, argmax=dev(arg), rev=rev)
    assert_terms_close(host(dx), rdx, rdxa, what=f"direct boundary {reducer} dx E={num_edges}")
    assert_terms_close(host(dw), rdw, rdwa, what=f"direct boundary {reducer} dw E={num_edges}")
