"""The allocation-free CSR forward (fixed per-device workspace) against the forward with a caller
workspace, through the C ABI: bit-identical results (same plan, same kernels) for two calls in a
row, the second on a smaller relation, for the sum and the max reducer; both also within the
oracle's bound.  An oversized relation is refused on the host before anything is enqueued."""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
from tests.parity import assert_terms_close

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def graph(n, F, seed, big=()):
    rng = np.random.default_rng(seed)
    deg = rng.choice([0, 1, 3, 8, 16, 17, 40, 200, 1500], size=n, p=[.1, .15, .15, .15, .1, .1, .1, .1, .05])
    for k, b in enumerate(big):
        deg[(k * 7919) % n] = b
    rp = np.zeros(n + 1, np.int64)
    np.cumsum(deg, out=rp[1:])
    E = int(rp[-1])
    col = rng.integers(0, n, E).astype(np.int32)
    x = rng.standard_normal((n, F)).astype(np.float32)
    w = rng.random(E).astype(np.float32)
    return rp, col, x, w


def call_noalloc(lib, rel, x, w, reducer, y, arg):
    return lib.load().tiga_mp_csr_fwd_noalloc(rel.ref, x.shape[1], lib._ptr(x), lib.MSG_EDGE_SCALED_SRC,
                                              lib._ptr(w), reducer, lib._ptr(y), lib._ptr(arg), lib._stream())


@pytest.mark.parametrize("reducer", ["sum", "max"])
def test_noalloc_forward_equals_workspace_forward(lib, reducer):
    red = lib.REDUCE_SUM if reducer == "sum" else lib.REDUCE_MAX
    # the second relation is smaller: the array keeps the first call's contents, which the second
    # call's plan overwrites where it reads
    for n, F, seed, big in [(9000, 16, 1, (60_000, 5000)), (3000, 32, 2, (12_000,))]:
        rp, col, x, w = graph(n, F, seed, big)
        assert rp[-1] > (1 << 16)   # the planned traversal (plan + gather + merge) runs
        rel = lib.Csr(dev(rp), dev(col), n)
        xd, wd = dev(x), dev(w)
        y = torch.full((n, F), float("nan"), device="cuda")
        arg = torch.full((n, F), -7, dtype=torch.int32, device="cuda") if red == lib.REDUCE_MAX else None
        assert call_noalloc(lib, rel, xd, wd, red, y, arg) == lib.TIGA_OK, lib.load().tiga_last_error()
        ref_y, ref_arg = lib.tiga_mp_csr_fwd(rel, xd, wd, reducer=red)
        torch.cuda.synchronize()
        assert torch.equal(y, ref_y)
        if red == lib.REDUCE_MAX:
            assert torch.equal(arg, ref_arg)
            oy, oarg = oracle.csr_max_fwd(rp, col, x, w)
            assert np.array_equal(arg.cpu().numpy(), oarg)
            assert np.array_equal(y.cpu().numpy().view(np.uint32), oy.view(np.uint32))
        else:
            oy, oya = oracle.csr_sum_fwd(rp, col, x, w)
            assert_terms_close(y.cpu().numpy(), oy, oya, what=f"noalloc y n={n}")


def test_noalloc_refuses_an_oversized_relation(lib):
    from paper_2609_24802_amd.binding import _Csr
    big = _Csr(50_000_000, 50_000_000, 1_000_000_000, 0x1000, 0x2000)
    fake = C.c_void_p(0x10000)
    L = lib.load()
    assert L.tiga_mp_csr_fwd_workspace(C.byref(big), 16, lib.REDUCE_SUM) > L.tiga_mp_csr_fwd_noalloc_limit()
    rc = L.tiga_mp_csr_fwd_noalloc(C.byref(big), 16, fake, lib.MSG_EDGE_SCALED_SRC, fake, lib.REDUCE_SUM, fake, None,
                                   None)
    assert rc == lib.TIGA_EUNSUPPORTED
    assert b"allocation-free" in L.tiga_last_error()
    assert L.tiga_mp_csr_fwd_noalloc_limit() == 64 << 20
