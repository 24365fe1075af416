"""The C-ABI library loads and exports every declared entry point, and its
host-side argument checks reject bad calls before anything reaches a device.

No compute call is made here: every call below returns from the host checks.
"""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tiga_mp.h")
LIB = os.path.join(ROOT, "paper_2609_24802_amd", "libtiga_mp.so")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b((?:tiga)_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def clib():
    if not os.path.exists(LIB):
        import __graft_entry__
        __graft_entry__.build()
    from paper_2609_24802_amd import binding
    return binding.load(LIB)


def test_exports_every_declared_symbol(clib):
    names = declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(clib, n), n


def test_abi_version(clib):
    assert clib.tiga_mp_abi_version() == 2


def test_struct_layouts_match_the_header(tmp_path):
    """The binding's ctypes structs have the header's field offsets and sizes (a C program compiled
    against include/tiga_mp.h prints them): the relation is (num_dst, num_src, num_edges, row_ptr,
    col_idx) and the reverse incidence is exactly (src_ptr, edge_id)."""
    import subprocess
    from paper_2609_24802_amd.binding import _Csr, _CsrT
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stdio.h>\n#include <stddef.h>\n#include "tiga_mp.h"\n'
        'int main(void) {\n'
        '  printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(tiga_csr), offsetof(tiga_csr, num_dst),\n'
        '         offsetof(tiga_csr, num_src), offsetof(tiga_csr, num_edges), offsetof(tiga_csr, row_ptr),\n'
        '         offsetof(tiga_csr, col_idx));\n'
        '  printf("%zu %zu %zu\\n", sizeof(tiga_csr_t), offsetof(tiga_csr_t, src_ptr), offsetof(tiga_csr_t, edge_id));\n'
        '  return 0;\n}\n')
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    out = subprocess.check_output([str(exe)]).decode().split("\n")
    csr = [int(v) for v in out[0].split()]
    rev = [int(v) for v in out[1].split()]
    assert csr == [C.sizeof(_Csr)] + [getattr(_Csr, f).offset for f in
                                      ("num_dst", "num_src", "num_edges", "row_ptr", "col_idx")]
    assert rev == [C.sizeof(_CsrT), _CsrT.src_ptr.offset, _CsrT.edge_id.offset]
    assert rev == [16, 0, 8] and [f for f, _ in _CsrT._fields_] == ["src_ptr", "edge_id"]


def _csr(num_dst, num_src, num_edges, rp=0x1000, col=0x2000):
    from paper_2609_24802_amd.binding import _Csr
    return _Csr(num_dst, num_src, num_edges, rp, col)


def test_csr_forward_argument_errors(clib):
    from paper_2609_24802_amd import binding as b
    fake = C.c_void_p(0x10000)
    rel = _csr(4, 4, 10)
    ws_need = clib.tiga_mp_csr_fwd_workspace(C.byref(rel), 16, b.REDUCE_SUM)
    assert ws_need > 0
    cases = [
        (dict(rel=None), b.TIGA_EINVAL),
        (dict(feat=0), b.TIGA_EINVAL),
        (dict(reducer=7), b.TIGA_EINVAL),
        (dict(msg=b.MSG_SRC), b.TIGA_EINVAL),  # weights given with an unweighted message
        (dict(w=None), b.TIGA_EINVAL),  # weighted message without weights
        (dict(y=None), b.TIGA_EINVAL),
        (dict(reducer=b.REDUCE_MAX), b.TIGA_EINVAL),  # max without argmax
        (dict(argmax=fake), b.TIGA_EINVAL),  # argmax with sum
        (dict(ws_bytes=16), b.TIGA_EWORKSPACE),
        (dict(ws=C.c_void_p(0x10010)), b.TIGA_EINVAL),  # misaligned workspace
        (dict(rel=_csr(4, 4, 3 << 30), reducer=b.REDUCE_MAX, argmax=fake), b.TIGA_EUNSUPPORTED),
        (dict(rel=_csr(-1, 4, 10)), b.TIGA_EINVAL),
        (dict(rel=_csr(4, 0, 10)), b.TIGA_EINVAL),
        (dict(rel=_csr(4, 4, 10, rp=0)), b.TIGA_EINVAL),
    ]
    for over, code in cases:
        a = dict(rel=rel, feat=16, x=fake, msg=b.MSG_EDGE_SCALED_SRC, w=fake, reducer=b.REDUCE_SUM, y=fake,
                 argmax=None, ws=fake, ws_bytes=1 << 40)
        a.update(over)
        relp = C.byref(a["rel"]) if a["rel"] is not None else None
        rc = clib.tiga_mp_csr_fwd(relp, a["feat"], a["x"], a["msg"], a["w"], a["reducer"], a["y"], a["argmax"],
                                  a["ws"], a["ws_bytes"], None)
        assert rc == code, (over, rc, clib.tiga_last_error())
        assert clib.tiga_last_error()


def test_csr_backward_and_transpose_errors(clib):
    from paper_2609_24802_amd import binding as b
    fake = C.c_void_p(0x10000)
    rel = _csr(4, 4, 10)
    rc = clib.tiga_mp_csr_bwd(C.byref(rel), None, 8, fake, b.MSG_SRC, None, b.REDUCE_SUM, None, fake, fake, fake,
                              fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL  # dw needs the weighted message
    rc = clib.tiga_mp_csr_bwd(C.byref(rel), None, 8, fake, b.MSG_EDGE_SCALED_SRC, fake, b.REDUCE_MAX, None, fake,
                              fake, None, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL  # max without argmax
    big = _csr(4, 4, 3 << 30)
    rc = clib.tiga_csr_transpose(C.byref(big), fake, fake, fake, 1 << 40, None)
    assert rc == b.TIGA_EUNSUPPORTED
    rc = clib.tiga_csr_transpose(C.byref(rel), fake, None, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL and b"edge_id" in clib.tiga_last_error()
    rc = clib.tiga_csr_validate(C.byref(rel), 3, None)
    assert rc == b.TIGA_EINVAL
    assert clib.tiga_csr_validate(C.byref(rel), 1, None) == b.TIGA_OK
    assert clib.tiga_csr_validate(C.byref(_csr(4, 0, 10)), 1, None) == b.TIGA_EGRAPH


def test_radius_dense_errors(clib):
    from paper_2609_24802_amd import binding as b
    fake = C.c_void_p(0x10000)
    rc = clib.tiga_mp_radius_fwd(100, 8, fake, fake, 0.1, 0.05, b.REDUCE_MAX, fake, None, fake, 1 << 40, None)
    assert rc == b.TIGA_EUNSUPPORTED
    rc = clib.tiga_mp_radius_fwd(100, 8, fake, fake, -0.1, 0.05, b.REDUCE_SUM, fake, None, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL
    rc = clib.tiga_mp_radius_fwd(100, 8, fake, fake, 0.1, 0.05, b.REDUCE_SUM, fake, None, fake, 8, None)
    assert rc == b.TIGA_EWORKSPACE
    rc = clib.tiga_mp_radius_bwd(100, 8, fake, None, 0.1, 0.05, fake, fake, fake, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL  # dpos needs x
    # 2 / sigma^2 must be finite in fp32 (else a coincident pair's weight would be NaN)
    rc = clib.tiga_mp_radius_fwd(100, 8, fake, fake, 0.1, 1e-20, b.REDUCE_SUM, fake, None, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL and b"sigma" in clib.tiga_last_error()
    rc = clib.tiga_mp_radius_bwd(100, 8, fake, fake, 0.1, 1e-20, fake, fake, fake, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL and b"sigma" in clib.tiga_last_error()
    rc = clib.tiga_mp_dense_fwd(100, fake, fake, 0.0, b.REDUCE_SUM, fake, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL
    rc = clib.tiga_mp_dense_fwd(100, fake, fake, 0.01, b.REDUCE_MAX, fake, fake, 1 << 40, None)
    assert rc == b.TIGA_EUNSUPPORTED
    rc = clib.tiga_mp_dense_fwd(100, fake, fake, 1e-20, b.REDUCE_SUM, fake, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL and b"normal" in clib.tiga_last_error()   # eps^2 underflows in fp32
    rc = clib.tiga_mp_dense_fwd(100, fake, fake, 1e20, b.REDUCE_SUM, fake, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL   # eps^2 overflows in fp32
    # feat 0 computes counts only, so count is required
    rc = clib.tiga_mp_radius_fwd(100, 0, fake, None, 0.1, 0.05, b.REDUCE_SUM, None, None, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL and b"count" in clib.tiga_last_error()
    rc = clib.tiga_mp_radius_fwd(100, -1, fake, None, 0.1, 0.05, b.REDUCE_SUM, None, fake, fake, 1 << 40, None)
    assert rc == b.TIGA_EINVAL
    # neighbour lists: nbr_ptr and nbr_idx are required, the workspace is checked
    assert clib.tiga_radius_neighbors(100, fake, 0.1, None, fake, fake, 1 << 40, None) == b.TIGA_EINVAL
    assert clib.tiga_radius_neighbors(100, fake, 0.1, fake, None, fake, 1 << 40, None) == b.TIGA_EINVAL
    assert clib.tiga_radius_neighbors(100, fake, 0.1, fake, fake, fake, 8, None) == b.TIGA_EWORKSPACE
    assert clib.tiga_radius_neighbors(0, None, 0.1, None, None, None, 0, None) == b.TIGA_OK
    # empty inputs are valid no-ops
    assert clib.tiga_mp_dense_fwd(0, None, None, 0.01, b.REDUCE_SUM, None, None, 0, None) == b.TIGA_OK
    assert clib.tiga_mp_radius_fwd(0, 8, None, None, 0.1, 0.05, b.REDUCE_SUM, None, None, None, 0, None) == b.TIGA_OK


def test_workspace_queries_monotone(clib):
    from paper_2609_24802_amd import binding as b
    small = clib.tiga_mp_csr_fwd_workspace(C.byref(_csr(1000, 1000, 16000)), 64, b.REDUCE_MAX)
    large = clib.tiga_mp_csr_fwd_workspace(C.byref(_csr(1_000_000, 1_000_000, 16_000_000)), 64, b.REDUCE_MAX)
    assert 0 < small < large
    assert clib.tiga_mp_radius_workspace(1000, 32) < clib.tiga_mp_radius_workspace(100000, 32)
    assert clib.tiga_mp_dense_workspace(65536) > 65536 * 16


def test_attention_errors(clib):
    from paper_2609_24802_amd import binding as b
    fake = C.c_void_p(0x10000)
    odd = C.c_void_p(0x10008)

    def call(n=100, heads=2, width=64, dt=b.DT_F16, q=fake, k=fake, v=fake, scale=0.125, rel=b.REL_TRIANGULAR,
             y=fake, lse=None):
        return clib.tiga_mp_attention_fwd(n, heads, width, dt, q, k, v, scale, rel, y, lse, None)

    assert call(width=96) == b.TIGA_EUNSUPPORTED
    assert call(width=256) == b.TIGA_EUNSUPPORTED
    assert call(n=1 << 31) == b.TIGA_EUNSUPPORTED
    assert call(n=1 << 30, heads=1 << 10) == b.TIGA_EUNSUPPORTED
    assert call(n=-1) == b.TIGA_EINVAL
    assert call(dt=7) == b.TIGA_EINVAL
    assert call(rel=5) == b.TIGA_EINVAL
    assert call(scale=0.0) == b.TIGA_EINVAL
    assert call(scale=-1.0) == b.TIGA_EINVAL
    assert call(scale=float("inf")) == b.TIGA_EINVAL
    assert call(scale=float("nan")) == b.TIGA_EINVAL
    assert call(v=None) == b.TIGA_EINVAL
    assert call(y=odd) == b.TIGA_EINVAL
    assert call(k=odd) == b.TIGA_EINVAL
    assert b"16-byte" in clib.tiga_last_error()
    # empty problems are valid no-ops
    assert call(n=0, q=None, k=None, v=None, y=None) == b.TIGA_OK
    assert call(heads=0, q=None, k=None, v=None, y=None) == b.TIGA_OK


def test_knn_errors(clib):
    from paper_2609_24802_amd import binding as b
    fake = C.c_void_p(0x10000)
    big = 1 << 40
    assert clib.tiga_mp_knn_fwd(100, 1, fake, fake, 33, b.REDUCE_SUM, fake, None, fake, big, None) == b.TIGA_EUNSUPPORTED
    assert clib.tiga_mp_knn_fwd(100, 1, fake, fake, -1, b.REDUCE_SUM, fake, None, fake, big, None) == b.TIGA_EINVAL
    assert clib.tiga_mp_knn_fwd(100, 1, fake, fake, 16, b.REDUCE_MAX, fake, None, fake, big, None) == b.TIGA_EUNSUPPORTED
    assert clib.tiga_mp_knn_fwd(100, 1, fake, None, 16, b.REDUCE_SUM, fake, None, fake, big, None) == b.TIGA_EINVAL
    assert clib.tiga_mp_knn_fwd(100, 1, fake, fake, 16, b.REDUCE_SUM, fake, None, fake, 8, None) == b.TIGA_EWORKSPACE
    assert clib.tiga_mp_knn_fwd(-1, 1, fake, fake, 16, b.REDUCE_SUM, fake, None, fake, big, None) == b.TIGA_EINVAL
    assert clib.tiga_mp_knn_fwd(0, 1, None, None, 16, b.REDUCE_SUM, None, None, None, 0, None) == b.TIGA_OK
    assert clib.tiga_mp_knn_workspace(1000) < clib.tiga_mp_knn_workspace(100000)


def test_edgenn_errors(clib):
    from paper_2609_24802_amd import binding as b
    f = C.c_void_p(0x10000)
    big = 1 << 40
    call = lambda n=100, F=8, H=32, O=3, r=0.1, ws=f, wsb=big: clib.tiga_mp_edgenn_fwd(
        n, F, H, O, f, f, r, f, f, f, f, f, ws, wsb, None)
    assert call(F=65) == b.TIGA_EUNSUPPORTED
    assert call(H=65) == b.TIGA_EUNSUPPORTED
    assert call(O=9) == b.TIGA_EUNSUPPORTED
    assert call(H=0) == b.TIGA_EINVAL
    assert call(r=0.0) == b.TIGA_EINVAL
    assert call(wsb=8) == b.TIGA_EWORKSPACE
    assert call(n=300_000_000) == b.TIGA_EUNSUPPORTED   # the shared cell directory's int32 keys
    assert call(n=0, ws=None, wsb=0) == b.TIGA_OK
    assert clib.tiga_mp_edgenn_bwd(100, 8, 32, 3, f, f, 0.1, f, f, f, f, None, f, f, f, f, f, f, f, big,
                                   None) == b.TIGA_EINVAL   # dy is required
    assert clib.tiga_mp_edgenn_workspace(1000, 8, 32, 3) < clib.tiga_mp_edgenn_workspace(100000, 8, 32, 3)


def test_csr_paged_host_checks(clib):
    """The paged forward reads row_ptr on the host: bad metadata and too-long rows are rejected there."""
    import numpy as np
    from paper_2609_24802_amd import binding as b
    from paper_2609_24802_amd.binding import _Csr
    fake = C.c_void_p(0x10000)
    rp = np.array([0, 3, 3, 10], np.int64)
    col = np.zeros(10, np.int32)
    rel = _Csr(3, 5, 10, rp.ctypes.data, col.ctypes.data)
    need = clib.tiga_mp_csr_fwd_paged_workspace(4, b.REDUCE_SUM, 8)
    assert need > 0
    rc = clib.tiga_mp_csr_fwd_paged(C.byref(rel), 4, fake, b.MSG_SRC, None, b.REDUCE_SUM, fake, None, 4, fake,
                                    1 << 40, None)
    assert rc == b.TIGA_EUNSUPPORTED and b"more than page_edges" in clib.tiga_last_error()
    bad = np.array([0, 3, 2, 10], np.int64)
    rel_bad = _Csr(3, 5, 10, bad.ctypes.data, col.ctypes.data)
    rc = clib.tiga_mp_csr_fwd_paged(C.byref(rel_bad), 4, fake, b.MSG_SRC, None, b.REDUCE_SUM, fake, None, 16, fake,
                                    1 << 40, None)
    assert rc == b.TIGA_EGRAPH
    rc = clib.tiga_mp_csr_fwd_paged(C.byref(rel), 4, fake, b.MSG_SRC, None, b.REDUCE_SUM, fake, None, 0, fake,
                                    1 << 40, None)
    assert rc == b.TIGA_EINVAL
