"""GPU parity of the paged CSR forward (relation in pinned host memory, staged page by page).

The pages run the resident gather-reduce on whole rows, so the paged result must equal the
resident one bit for bit (y, and argmax in global edge positions), and both match the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_24802_amd import synth
from tests.parity import assert_terms_close

pytestmark = pytest.mark.gpu


def pinned(a):
    return torch.from_numpy(np.ascontiguousarray(a)).pin_memory()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def graphs():
    g1 = synth.csr_uniform_small()
    g2 = synth.csr_powerlaw(20000, 400000, 16, cap=5000, cfg=21, with_dy=False)
    # empty rows at the start, the middle and the end, and one heavy row
    rng = np.random.default_rng(4)
    deg = rng.integers(0, 12, 3000)
    deg[:5] = 0
    deg[1500:1510] = 0
    deg[-7:] = 0
    deg[777] = 2500
    rp = np.zeros(3001, np.int64)
    np.cumsum(deg, out=rp[1:])
    e = int(rp[-1])
    g3 = dict(row_ptr=rp, col=rng.integers(0, 3000, e).astype(np.int32),
              w=rng.random(e, dtype=np.float32), x=rng.standard_normal((3000, 12)).astype(np.float32),
              num_dst=3000, num_src=3000)
    return {"uniform": g1, "powerlaw": g2, "empty_rows": g3}


GRAPHS = graphs()


@pytest.mark.parametrize("name", list(GRAPHS))
@pytest.mark.parametrize("reducer", ["sum", "max"])
@pytest.mark.parametrize("weighted", [True, False])
def test_paged_equals_resident(lib, name, reducer, weighted):
    g = GRAPHS[name]
    rp, col, x, w = g["row_ptr"], g["col"], g["x"], g["w"]
    red = lib.REDUCE_SUM if reducer == "sum" else lib.REDUCE_MAX
    maxdeg = int(np.diff(rp).max())
    rel_d = lib.Csr(dev(rp), dev(col), g["num_src"])
    y_r, a_r = lib.tiga_mp_csr_fwd(rel_d, dev(x), dev(w) if weighted else None, reducer=red)
    rel_h = lib.HostCsr(pinned(rp), pinned(col), g["num_src"])
    for page in (maxdeg, maxdeg + 1, 4 * maxdeg + 3, int(rp[-1]) + 1):
        y_p, a_p = lib.tiga_mp_csr_fwd_paged(rel_h, dev(x), pinned(w) if weighted else None, reducer=red,
                                             page_edges=page)
        torch.cuda.synchronize()
        assert torch.equal(y_p, y_r), (name, page)
        if red == lib.REDUCE_MAX:
            assert torch.equal(a_p, a_r), (name, page)
    if red == lib.REDUCE_SUM:
        ry, rya = oracle.csr_sum_fwd(rp, col, x, w if weighted else None)
        assert_terms_close(y_p.cpu().numpy(), ry, rya, what="paged sum")
    else:
        ry, rarg = oracle.csr_max_fwd(rp, col, x, w if weighted else None)
        assert np.array_equal(y_p.cpu().numpy(), ry) and np.array_equal(a_p.cpu().numpy(), rarg)


def test_paged_rejects_a_row_longer_than_a_page(lib):
    g = GRAPHS["empty_rows"]
    rel_h = lib.HostCsr(pinned(g["row_ptr"]), pinned(g["col"]), g["num_src"])
    with pytest.raises(lib.TigaError) as e:
        lib.tiga_mp_csr_fwd_paged(rel_h, dev(g["x"]), pinned(g["w"]), page_edges=2499)
    assert e.value.code == lib.TIGA_EUNSUPPORTED
