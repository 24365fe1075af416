"""CPU oracle for fused message passing -- test infrastructure only.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or runs it.

The numerics live in ``tiga_oracle.c`` (plain C, OpenMP over independent
outputs, fp64 accumulation); this module is argument marshalling with numpy.
Every sum comes back as fp64 together with the per-output sum of absolute
term values, so a caller can check an fp32 result of any summation order
against ``|got - ref| <= rtol * sum|terms|``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tiga_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libtiga_oracle.so")
_lock = threading.Lock()
_lib = None

CFLAGS = ["-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
          "-shared", "-fPIC", "-Wall"]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no contraction, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = C.CDLL(build())
            i64, i32, vp, f32 = C.c_int64, C.c_int32, C.c_void_p, C.c_float
            sig = {
                "tiga_oracle_threads": (C.c_int, []),
                "tiga_oracle_set_threads": (None, [C.c_int]),
                "tiga_oracle_csr_sum_fwd": (None, [i64, vp, i32, vp, vp, vp, vp, vp, vp]),
                "tiga_oracle_csr_max_fwd": (None, [i64, vp, i32, vp, vp, vp, vp, vp, vp]),
                "tiga_oracle_csr_sum_bwd": (None, [i64, i64, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
                "tiga_oracle_csr_max_bwd": (None, [i64, i64, i64, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
                "tiga_oracle_radius_fwd": (C.c_int, [i64, i32, vp, vp, f32, f32, i64, vp, vp, vp, vp]),
                "tiga_oracle_radius_bwd": (C.c_int, [i64, i32, vp, vp, vp, f32, f32, i64, vp, vp, vp, vp, vp]),
                "tiga_oracle_radius_neighbors": (C.c_int, [i64, vp, f32, i64, vp, vp, vp, vp]),
                "tiga_oracle_dense_fwd": (None, [i64, vp, vp, f32, i64, vp, vp, vp]),
                "tiga_oracle_edgenn": (None, [i64, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
                "tiga_oracle_knn": (C.c_int, [i64, i32, vp, vp, i32, i64, vp, vp, vp, vp]),
                "tiga_oracle_f16_to_double": (C.c_double, [C.c_uint16]),
                "tiga_oracle_bf16_to_double": (C.c_double, [C.c_uint16]),
                "tiga_oracle_attention_fwd": (C.c_int, [i64, i32, i32, C.c_int, vp, vp, vp, C.c_double,
                                                        C.c_int, i64, vp, vp, vp, vp]),
            }
            for name, (res, args) in sig.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def threads() -> int:
    return int(_load().tiga_oracle_threads())


def set_threads(n: int) -> None:
    """Threads for later calls (n <= 0: all host cores again); results do not depend on it."""
    _load().tiga_oracle_set_threads(int(n))


def _rows(rows, n):
    if rows is None:
        return None, n
    rows = _c(rows, np.int64).reshape(-1)
    return rows, rows.shape[0]


def csr_sum_fwd(row_ptr, col, x, w=None, rows=None):
    """Weighted-sum forward; returns (y fp64 [nrows,F], sum|terms| fp64)."""
    row_ptr, col, x, w = _c(row_ptr, np.int64), _c(col, np.int32), _c(x, np.float32), _c(w, np.float32)
    F = x.shape[1]
    rows, nrows = _rows(rows, row_ptr.shape[0] - 1)
    y = np.empty((nrows, F), np.float64)
    ya = np.empty((nrows, F), np.float64)
    _load().tiga_oracle_csr_sum_fwd(nrows, _p(rows), F, _p(row_ptr), _p(col), _p(x), _p(w), _p(y), _p(ya))
    return y, ya


def csr_max_fwd(row_ptr, col, x, w=None, rows=None):
    """Max forward; returns (y fp32 [nrows,F], argmax int32 [nrows,F])."""
    row_ptr, col, x, w = _c(row_ptr, np.int64), _c(col, np.int32), _c(x, np.float32), _c(w, np.float32)
    F = x.shape[1]
    rows, nrows = _rows(rows, row_ptr.shape[0] - 1)
    y = np.empty((nrows, F), np.float32)
    arg = np.empty((nrows, F), np.int32)
    _load().tiga_oracle_csr_max_fwd(nrows, _p(rows), F, _p(row_ptr), _p(col), _p(x), _p(w), _p(y), _p(arg))
    return y, arg


def csr_sum_bwd(row_ptr, col, x, w, dy, num_src, want_dx=True, want_dw=True):
    """Weighted-sum VJP; returns (dx, dx_abs, dw, dw_abs), fp64 (None where not requested)."""
    row_ptr, col, x, w, dy = (_c(row_ptr, np.int64), _c(col, np.int32), _c(x, np.float32),
                              _c(w, np.float32), _c(dy, np.float32))
    F = dy.shape[1]
    E = col.shape[0]
    dx = np.empty((num_src, F), np.float64) if want_dx else None
    dxa = np.empty((num_src, F), np.float64) if want_dx else None
    dw = np.empty(E, np.float64) if want_dw else None
    dwa = np.empty(E, np.float64) if want_dw else None
    _load().tiga_oracle_csr_sum_bwd(row_ptr.shape[0] - 1, num_src, F, _p(row_ptr), _p(col), _p(x),
                                    _p(w), _p(dy), _p(dx), _p(dxa), _p(dw), _p(dwa))
    return dx, dxa, dw, dwa


def csr_max_bwd(row_ptr, col, x, w, arg, dy, num_src, want_dx=True, want_dw=True):
    """Max VJP routed through argmax; returns (dx, dx_abs, dw, dw_abs), fp64."""
    row_ptr, col, x, w, arg, dy = (_c(row_ptr, np.int64), _c(col, np.int32), _c(x, np.float32),
                                   _c(w, np.float32), _c(arg, np.int32), _c(dy, np.float32))
    F = dy.shape[1]
    E = col.shape[0]
    dx = np.empty((num_src, F), np.float64) if want_dx else None
    dxa = np.empty((num_src, F), np.float64) if want_dx else None
    dw = np.empty(E, np.float64) if want_dw else None
    dwa = np.empty(E, np.float64) if want_dw else None
    _load().tiga_oracle_csr_max_bwd(row_ptr.shape[0] - 1, num_src, E, F, _p(row_ptr), _p(col), _p(x),
                                    _p(w), _p(arg), _p(dy), _p(dx), _p(dxa), _p(dw), _p(dwa))
    return dx, dxa, dw, dwa


def radius_fwd(pos, x, radius, sigma, pts=None):
    """Radius forward; returns (y fp64 [npts,F], sum|terms|, count int32 [npts])."""
    pos, x = _c(pos, np.float32), _c(x, np.float32)
    n, F = x.shape
    pts, npts = _rows(pts, n)
    y = np.empty((npts, F), np.float64)
    ya = np.empty((npts, F), np.float64)
    cnt = np.empty(npts, np.int32)
    rc = _load().tiga_oracle_radius_fwd(n, F, _p(pos), _p(x), float(radius), float(sigma), npts,
                                        _p(pts), _p(y), _p(ya), _p(cnt))
    if rc != 0:
        raise MemoryError("oracle radius forward: allocation failed")
    return y, ya, cnt


def radius_bwd(pos, x, dy, radius, sigma, pts=None):
    """Radius VJP; returns (dx, dx_abs, dpos, dpos_abs), fp64, for the requested points."""
    pos, x, dy = _c(pos, np.float32), _c(x, np.float32), _c(dy, np.float32)
    n, F = x.shape
    pts, npts = _rows(pts, n)
    dx = np.empty((npts, F), np.float64)
    dxa = np.empty((npts, F), np.float64)
    dp = np.empty((npts, 3), np.float64)
    dpa = np.empty((npts, 3), np.float64)
    rc = _load().tiga_oracle_radius_bwd(n, F, _p(pos), _p(x), _p(dy), float(radius), float(sigma),
                                        npts, _p(pts), _p(dx), _p(dxa), _p(dp), _p(dpa))
    if rc != 0:
        raise MemoryError("oracle radius backward: allocation failed")
    return dx, dxa, dp, dpa


def radius_neighbors(pos, radius, pts=None):
    """Accepted neighbour lists (ascending); returns (ptr int64 [npts+1], idx int32)."""
    pos = _c(pos, np.float32)
    n = pos.shape[0]
    pts, npts = _rows(pts, n)
    cnt = np.empty(npts, np.int32)
    lib = _load()
    if lib.tiga_oracle_radius_neighbors(n, _p(pos), float(radius), npts, _p(pts), _p(cnt), None, None):
        raise MemoryError("oracle radius neighbours: allocation failed")
    ptr = np.zeros(npts + 1, np.int64)
    np.cumsum(cnt, out=ptr[1:])
    idx = np.empty(int(ptr[-1]), np.int32)
    if lib.tiga_oracle_radius_neighbors(n, _p(pos), float(radius), npts, _p(pts), None, _p(ptr), _p(idx)):
        raise MemoryError("oracle radius neighbours: allocation failed")
    return ptr, idx


def dense_fwd(pos, q, eps, pts=None):
    """Dense softened inverse-square sum; returns (y fp64 [npts,3], sum|terms|)."""
    pos, q = _c(pos, np.float32), _c(q, np.float32)
    n = pos.shape[0]
    pts, npts = _rows(pts, n)
    y = np.empty((npts, 3), np.float64)
    ya = np.empty((npts, 3), np.float64)
    _load().tiga_oracle_dense_fwd(n, _p(pos), _p(q), float(eps), npts, _p(pts), _p(y), _p(ya))
    return y, ya


_ATTN_DTYPES = {"f16": 0, "bf16": 1}
_ATTN_RELATIONS = {"triangular": 0, "dense": 1}


def half_to_double(bits, dtype):
    """Exact widening of 16-bit patterns (binary16 or bfloat16) to float64, one call per value."""
    fn = _load().tiga_oracle_f16_to_double if dtype == "f16" else _load().tiga_oracle_bf16_to_double
    bits = np.asarray(bits, np.uint16).reshape(-1)
    return np.array([fn(int(b)) for b in bits], np.float64)


def attention_fwd(q, k, v, scale, dtype="f16", relation="triangular", pts=None):
    """Online-softmax attention over a triangular (causal, diagonal included) or dense relation.

    q, k, v: uint16 bit patterns [H, n, D] (head-major).  Returns (y, yabs, lse): y and yabs fp64
    [npts, H, D] (yabs = sum_j p_ij |v_jd| with normalized weights p), lse fp64 [npts, H]."""
    q, k, v = (np.ascontiguousarray(a).view(np.uint16) for a in (q, k, v))
    H, n, D = q.shape
    pts, npts = _rows(pts, n)
    y = np.empty((npts, H, D), np.float64)
    ya = np.empty((npts, H, D), np.float64)
    lse = np.empty((npts, H), np.float64)
    rc = _load().tiga_oracle_attention_fwd(n, H, D, _ATTN_DTYPES[dtype], _p(q), _p(k), _p(v), float(scale),
                                           _ATTN_RELATIONS[relation], npts, _p(pts), _p(y), _p(ya), _p(lse))
    if rc != 0:
        raise ValueError("oracle attention: unknown dtype or relation")
    return y, ya, lse


def knn(pos, x, k, pts=None):
    """Exact kNN (self excluded, key (d2, index)); returns (nbr int32 [npts, k], y fp64 [npts, F], yabs)."""
    pos = _c(pos, np.float32).reshape(-1, 3)
    n = pos.shape[0]
    x = None if x is None else _c(x, np.float32).reshape(n, -1)
    F = 0 if x is None else x.shape[1]
    pts, npts = _rows(pts, n)
    nbr = np.empty((npts, k), np.int32)
    y = np.empty((npts, F), np.float64)
    ya = np.empty((npts, F), np.float64)
    if _load().tiga_oracle_knn(n, F, _p(pos), _p(x), int(k), npts, _p(pts), _p(nbr), _p(y), _p(ya)):
        raise MemoryError("oracle kNN: allocation failed")
    return nbr, y, ya


_EDGENN_OUTS = ("y", "dx", "dp", "dW1", "db1", "dW2", "db2")


def edgenn(pos, x, ptr, idx, W1, b1, W2, b2, dy=None, terms=False):
    """Edge-local MLP message summed per destination over the relation (ptr, idx); with dy also the
    gradients of <dy, y>.  Returns dict(y, dx, dp, dW1, db1, dW2, db2) in fp64.

    With terms=True returns (values, mag, slack), three such dicts: mag is each output's
    absolute-value evaluation with the oracle's ReLU decisions held (the error bound of any fp32
    evaluation order), slack what reaches the output through ReLU decisions fp32 cannot settle."""
    pos, x = _c(pos, np.float32).reshape(-1, 3), _c(x, np.float32)
    n = pos.shape[0]
    x = x.reshape(n, -1)
    F = x.shape[1]
    W1, b1, W2, b2 = (_c(a, np.float32) for a in (W1, b1, W2, b2))
    H, O = W1.shape[0], W2.shape[0]
    assert W1.shape == (H, 3 + F) and b1.shape == (H,) and W2.shape == (O, H) and b2.shape == (O,)
    ptr, idx = _c(ptr, np.int64), _c(idx, np.int32)
    dy = _c(dy, np.float32)
    shapes = dict(y=(n, O), dx=(n, F), dp=(n, 3), dW1=(H, 3 + F), db1=(H,), dW2=(O, H), db2=(O,))
    keys = _EDGENN_OUTS if dy is not None else ("y",)

    def outs():
        return {k: np.empty(shapes[k]) for k in keys}

    def table(d):
        return (C.c_void_p * 7)(*[_p(d.get(k)) for k in _EDGENN_OUTS])

    val = outs()
    mag = outs() if terms else None
    slack = outs() if terms else None
    tv = table(val)
    tm = table(mag) if terms else None
    ts = table(slack) if terms else None
    _load().tiga_oracle_edgenn(n, F, H, O, _p(pos), _p(x), _p(ptr), _p(idx), _p(W1), _p(b1), _p(W2), _p(b2),
                               _p(dy), tv, tm, ts)
    return (val, mag, slack) if terms else val
