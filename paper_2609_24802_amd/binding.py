"""Python binding of the gfx950 fused message-passing library (ctypes).

Argument marshalling only: every function below checks tensor shapes, dtypes
and devices, allocates outputs and the workspace with torch (device memory and
the current stream are the only things torch provides here), and calls the
C entry point of the same name.  All computation happens in the HIP kernels of
``libtiga_mp.so``; if that library is missing or cannot be loaded, every call
raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes as C
import os
import threading

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtiga_mp.so")

TIGA_OK, TIGA_EINVAL, TIGA_EGRAPH, TIGA_EUNSUPPORTED, TIGA_EWORKSPACE, TIGA_EDEVICE = 0, -1, -2, -3, -4, -5
REDUCE_SUM, REDUCE_MAX = 0, 1
MSG_SRC, MSG_EDGE_SCALED_SRC = 0, 1
DT_F16, DT_BF16 = 0, 1
REL_TRIANGULAR, REL_DENSE = 0, 1
_STATUS = {0: "TIGA_OK", -1: "TIGA_EINVAL", -2: "TIGA_EGRAPH", -3: "TIGA_EUNSUPPORTED",
           -4: "TIGA_EWORKSPACE", -5: "TIGA_EDEVICE"}


class TigaError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{_STATUS.get(code, code)}: {message}")
        self.code = code


class _Csr(C.Structure):
    _fields_ = [("num_dst", C.c_int64), ("num_src", C.c_int64), ("num_edges", C.c_int64),
                ("row_ptr", C.c_void_p), ("col_idx", C.c_void_p)]


class _CsrT(C.Structure):
    _fields_ = [("src_ptr", C.c_void_p), ("edge_id", C.c_void_p)]


_lib = None
_lock = threading.Lock()

_SIGS = {
    "tiga_last_error": (C.c_char_p, []),
    "tiga_mp_abi_version": (C.c_int, []),
    "tiga_mp_csr_fwd_workspace": (C.c_size_t, [C.c_void_p, C.c_int32, C.c_int]),
    "tiga_mp_csr_fwd": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_int, C.c_void_p, C.c_int, C.c_void_p,
                                  C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "tiga_mp_csr_fwd_noalloc_limit": (C.c_size_t, []),
    "tiga_mp_csr_fwd_noalloc": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_int, C.c_void_p, C.c_int,
                                          C.c_void_p, C.c_void_p, C.c_void_p]),
    "tiga_mp_csr_bwd_workspace": (C.c_size_t, [C.c_void_p, C.c_int32, C.c_int]),
    "tiga_mp_csr_bwd": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int, C.c_void_p, C.c_int,
                                  C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                  C.c_void_p]),
    "tiga_csr_transpose_workspace": (C.c_size_t, [C.c_void_p]),
    "tiga_csr_transpose": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "tiga_csr_validate": (C.c_int, [C.c_void_p, C.c_int, C.c_void_p]),
    "tiga_mp_radius_workspace": (C.c_size_t, [C.c_int64, C.c_int32]),
    "tiga_mp_radius_fwd": (C.c_int, [C.c_int64, C.c_int32, C.c_void_p, C.c_void_p, C.c_float, C.c_float, C.c_int,
                                     C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "tiga_mp_radius_bwd": (C.c_int, [C.c_int64, C.c_int32, C.c_void_p, C.c_void_p, C.c_float, C.c_float,
                                     C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "tiga_radius_neighbors": (C.c_int, [C.c_int64, C.c_void_p, C.c_float, C.c_void_p, C.c_void_p, C.c_void_p,
                                        C.c_size_t, C.c_void_p]),
    "tiga_mp_dense_workspace": (C.c_size_t, [C.c_int64]),
    "tiga_mp_dense_fwd": (C.c_int, [C.c_int64, C.c_void_p, C.c_void_p, C.c_float, C.c_int, C.c_void_p,
                                    C.c_void_p, C.c_size_t, C.c_void_p]),
    "tiga_mp_csr_fwd_paged_workspace": (C.c_size_t, [C.c_int32, C.c_int, C.c_int64]),
    "tiga_mp_csr_fwd_paged": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_int, C.c_void_p, C.c_int, C.c_void_p,
                                        C.c_void_p, C.c_int64, C.c_void_p, C.c_size_t, C.c_void_p]),
    "tiga_mp_edgenn_workspace": (C.c_size_t, [C.c_int64, C.c_int32, C.c_int32, C.c_int32]),
    "tiga_mp_edgenn_fwd": (C.c_int, [C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_float,
                                     C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                     C.c_size_t, C.c_void_p]),
    "tiga_mp_edgenn_bwd": (C.c_int, [C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_float,
                                     C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                     C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                     C.c_size_t, C.c_void_p]),
    "tiga_mp_knn_workspace": (C.c_size_t, [C.c_int64]),
    "tiga_mp_knn_fwd": (C.c_int, [C.c_int64, C.c_int32, C.c_void_p, C.c_void_p, C.c_int32, C.c_int, C.c_void_p,
                                  C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "tiga_mp_attention_fwd": (C.c_int, [C.c_int64, C.c_int32, C.c_int32, C.c_int, C.c_void_p, C.c_void_p,
                                        C.c_void_p, C.c_float, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p]),
    "tiga_mp_set_kernel_events": (C.c_int, [C.c_void_p, C.c_void_p]),
}


def load(path: str = LIB_PATH):
    """Load the HIP library (torch's HIP runtime is loaded first and shared)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(path):
                raise RuntimeError(f"HIP library not built: {path} is missing (run __graft_entry__.build())")
            lib = C.CDLL(path)
            for name, (res, args) in _SIGS.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
    return _lib


def _check(rc: int):
    if rc != TIGA_OK:
        raise TigaError(rc, load().tiga_last_error().decode())


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream():
    """The current HIP stream of the current device, as a void pointer.  torch's raw-stream
    accessor avoids building a Stream object (about 3 us per call); the public call is the
    fallback."""
    if _raw_stream is not None:
        return C.c_void_p(_raw_stream(torch.cuda.current_device()))
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, dtype, name, shape=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _workspace(nbytes: int, device):
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


class Csr:
    """A destination-major CSR relation on the device (row_ptr int64, col_idx int32)."""

    def __init__(self, row_ptr: torch.Tensor, col_idx: torch.Tensor, num_src: int):
        self.row_ptr = _dev(row_ptr, torch.int64, "row_ptr")
        self.col_idx = _dev(col_idx, torch.int32, "col_idx")
        self.num_dst = row_ptr.numel() - 1
        self.num_src = int(num_src)
        self.num_edges = col_idx.numel()
        self._c = _Csr(self.num_dst, self.num_src, self.num_edges, self.row_ptr.data_ptr(),
                       self.col_idx.data_ptr() if self.num_edges else None)

    @property
    def ref(self):
        return C.byref(self._c)


class CsrT:
    """Reverse incidence built by :func:`tiga_csr_transpose`."""

    def __init__(self, src_ptr, edge_id):
        self.src_ptr, self.edge_id = src_ptr, edge_id
        self._c = _CsrT(src_ptr.data_ptr(), edge_id.data_ptr() if edge_id.numel() else None)

    @property
    def ref(self):
        return C.byref(self._c)


def tiga_mp_abi_version() -> int:
    return int(load().tiga_mp_abi_version())


def tiga_mp_set_kernel_events(start=None, stop=None):
    """Arm hipEvents (torch.cuda.Event, already recorded once) around the next dominant kernel."""
    lib = load()
    s = C.c_void_p(start.cuda_event) if start is not None else None
    e = C.c_void_p(stop.cuda_event) if stop is not None else None
    _check(lib.tiga_mp_set_kernel_events(s, e))


def tiga_mp_csr_fwd(rel: Csr, x: torch.Tensor, w: torch.Tensor | None = None, reducer: int = REDUCE_SUM,
                    y: torch.Tensor | None = None, argmax: torch.Tensor | None = None, ws=None):
    """Fused forward over a stored CSR relation; returns (y, argmax or None)."""
    lib = load()
    feat = x.shape[1]
    _dev(x, torch.float32, "x", (rel.num_src, feat))
    msg = MSG_SRC
    if w is not None:
        _dev(w, torch.float32, "w", (rel.num_edges,))
        msg = MSG_EDGE_SCALED_SRC
    if y is None:
        y = torch.empty(rel.num_dst, feat, dtype=torch.float32, device=x.device)
    if reducer == REDUCE_MAX and argmax is None:
        argmax = torch.empty(rel.num_dst, feat, dtype=torch.int32, device=x.device)
    need = lib.tiga_mp_csr_fwd_workspace(rel.ref, feat, reducer)
    if ws is None:
        ws = _workspace(need, x.device)
    _check(lib.tiga_mp_csr_fwd(rel.ref, feat, _ptr(x), msg, _ptr(w), reducer, _ptr(y), _ptr(argmax),
                               _ptr(ws), ws.numel(), _stream()))
    return y, argmax


def tiga_mp_csr_fwd_noalloc(rel: Csr, x: torch.Tensor, w: torch.Tensor | None = None, reducer: int = REDUCE_SUM,
                            y: torch.Tensor | None = None, argmax: torch.Tensor | None = None):
    """tiga_mp_csr_fwd without a workspace (the library's fixed per-device array); pass y (and argmax)
    to make the whole call allocation-free.  Returns (y, argmax or None)."""
    lib = load()
    feat = x.shape[1]
    _dev(x, torch.float32, "x", (rel.num_src, feat))
    msg = MSG_SRC
    if w is not None:
        _dev(w, torch.float32, "w", (rel.num_edges,))
        msg = MSG_EDGE_SCALED_SRC
    if y is None:
        y = torch.empty(rel.num_dst, feat, dtype=torch.float32, device=x.device)
    if reducer == REDUCE_MAX and argmax is None:
        argmax = torch.empty(rel.num_dst, feat, dtype=torch.int32, device=x.device)
    _check(lib.tiga_mp_csr_fwd_noalloc(rel.ref, feat, _ptr(x), msg, _ptr(w), reducer, _ptr(y), _ptr(argmax),
                                       _stream()))
    return y, argmax


def _host(t, dtype, name, n=None):
    if not isinstance(t, torch.Tensor) or t.is_cuda:
        raise TypeError(f"{name} must be a host (CPU) tensor")
    if t.dtype != dtype or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous {dtype} host tensor")
    if n is not None and t.numel() != n:
        raise ValueError(f"{name} has {t.numel()} entries, expected {n}")
    return t


class HostCsr:
    """A destination-major CSR relation kept in host memory (pin it for asynchronous copies)."""

    def __init__(self, row_ptr: torch.Tensor, col_idx: torch.Tensor, num_src: int):
        self.row_ptr = _host(row_ptr, torch.int64, "row_ptr")
        self.col_idx = _host(col_idx, torch.int32, "col_idx")
        self.num_dst = row_ptr.numel() - 1
        self.num_src = int(num_src)
        self.num_edges = col_idx.numel()
        self._c = _Csr(self.num_dst, self.num_src, self.num_edges, self.row_ptr.data_ptr(),
                       self.col_idx.data_ptr() if self.num_edges else None)

    @property
    def ref(self):
        return C.byref(self._c)


def tiga_mp_csr_fwd_paged(rel: HostCsr, x: torch.Tensor, w: torch.Tensor | None = None, reducer: int = REDUCE_SUM,
                          page_edges: int = 1 << 24, ws=None):
    """tiga_mp_csr_fwd with the relation (and w) in host memory, staged in pages of whole rows with at most
    page_edges edges; x and the outputs on the device.  Returns (y, argmax or None)."""
    lib = load()
    feat = x.shape[1]
    _dev(x, torch.float32, "x", (rel.num_src, feat))
    msg = MSG_SRC
    if w is not None:
        _host(w, torch.float32, "w", rel.num_edges)
        msg = MSG_EDGE_SCALED_SRC
    y = torch.empty(rel.num_dst, feat, dtype=torch.float32, device=x.device)
    argmax = torch.empty(rel.num_dst, feat, dtype=torch.int32, device=x.device) if reducer == REDUCE_MAX else None
    if ws is None:
        ws = _workspace(lib.tiga_mp_csr_fwd_paged_workspace(feat, reducer, int(page_edges)), x.device)
    _check(lib.tiga_mp_csr_fwd_paged(rel.ref, feat, _ptr(x), msg, _ptr(w), reducer, _ptr(y), _ptr(argmax),
                                     int(page_edges), _ptr(ws), ws.numel(), _stream()))
    return y, argmax


def tiga_mp_csr_bwd(rel: Csr, dy: torch.Tensor, x: torch.Tensor | None = None, w: torch.Tensor | None = None,
                    reducer: int = REDUCE_SUM, argmax: torch.Tensor | None = None, rev: CsrT | None = None,
                    want_dx: bool = True, want_dw: bool = True, ws=None):
    """VJP of tiga_mp_csr_fwd; returns (dx or None, dw or None)."""
    lib = load()
    feat = dy.shape[1]
    _dev(dy, torch.float32, "dy", (rel.num_dst, feat))
    msg = MSG_EDGE_SCALED_SRC if w is not None else MSG_SRC
    want_dw = want_dw and w is not None
    dx = torch.empty(rel.num_src, feat, dtype=torch.float32, device=dy.device) if want_dx else None
    dw = torch.empty(rel.num_edges, dtype=torch.float32, device=dy.device) if want_dw else None
    need = lib.tiga_mp_csr_bwd_workspace(rel.ref, feat, reducer)
    if ws is None:
        ws = _workspace(need, dy.device)
    _check(lib.tiga_mp_csr_bwd(rel.ref, rev.ref if rev is not None else None, feat, _ptr(x), msg, _ptr(w),
                               reducer, _ptr(argmax), _ptr(dy), _ptr(dx), _ptr(dw), _ptr(ws), ws.numel(),
                               _stream()))
    return dx, dw


def tiga_csr_transpose(rel: Csr) -> CsrT:
    lib = load()
    dev = rel.row_ptr.device
    src_ptr = torch.empty(rel.num_src + 1, dtype=torch.int64, device=dev)
    edge_id = torch.empty(rel.num_edges, dtype=torch.int32, device=dev)
    ws = _workspace(lib.tiga_csr_transpose_workspace(rel.ref), dev)
    _check(lib.tiga_csr_transpose(rel.ref, _ptr(src_ptr), _ptr(edge_id) if rel.num_edges else None, _ptr(ws),
                                  ws.numel(), _stream()))
    return CsrT(src_ptr, edge_id)


def tiga_csr_validate(rel: Csr, level: int = 2):
    """Raise TigaError (TIGA_EGRAPH) on an invalid relation."""
    _check(load().tiga_csr_validate(rel.ref, level, _stream()))


def tiga_mp_radius_fwd(pos: torch.Tensor, x: torch.Tensor, radius: float, sigma: float, want_count: bool = True,
                       y=None, count=None, ws=None):
    lib = load()
    n, feat = x.shape
    _dev(pos, torch.float32, "pos", (n, 3))
    _dev(x, torch.float32, "x", (n, feat))
    if y is None:
        y = torch.empty(n, feat, dtype=torch.float32, device=x.device)
    if want_count and count is None:
        count = torch.empty(n, dtype=torch.int32, device=x.device)
    if ws is None:
        ws = _workspace(lib.tiga_mp_radius_workspace(n, feat), x.device)
    _check(lib.tiga_mp_radius_fwd(n, feat, _ptr(pos), _ptr(x), float(radius), float(sigma), REDUCE_SUM, _ptr(y),
                                  _ptr(count), _ptr(ws), ws.numel(), _stream()))
    return y, count


def tiga_mp_radius_bwd(pos, x, dy, radius: float, sigma: float, want_dx: bool = True, want_dpos: bool = True,
                       ws=None):
    lib = load()
    n, feat = dy.shape
    _dev(pos, torch.float32, "pos", (n, 3))
    _dev(dy, torch.float32, "dy", (n, feat))
    if want_dpos:
        _dev(x, torch.float32, "x", (n, feat))
    dx = torch.empty(n, feat, dtype=torch.float32, device=dy.device) if want_dx else None
    dpos = torch.empty(n, 3, dtype=torch.float32, device=dy.device) if want_dpos else None
    if ws is None:
        ws = _workspace(lib.tiga_mp_radius_workspace(n, feat), dy.device)
    _check(lib.tiga_mp_radius_bwd(n, feat, _ptr(pos), _ptr(x) if want_dpos else None, float(radius), float(sigma),
                                  _ptr(dy), _ptr(dx), _ptr(dpos), _ptr(ws), ws.numel(), _stream()))
    return dx, dpos


def tiga_radius_neighbors(pos: torch.Tensor, radius: float, count: torch.Tensor | None = None):
    """Accepted neighbour lists; returns (count int32, ptr int64 [n+1], idx int32).  Synchronizes.

    The two phases of the C call: the counts come from the forward with no features (or are
    passed in), their exclusive prefix sum is the caller's nbr_ptr, then the lists are filled."""
    lib = load()
    n = pos.shape[0]
    _dev(pos, torch.float32, "pos", (n, 3))
    ws = _workspace(lib.tiga_mp_radius_workspace(n, 0), pos.device)
    if count is None:
        count = torch.empty(n, dtype=torch.int32, device=pos.device)
        _check(lib.tiga_mp_radius_fwd(n, 0, _ptr(pos), None, float(radius), 1.0, REDUCE_SUM, None, _ptr(count),
                                      _ptr(ws), ws.numel(), _stream()))
    else:
        _dev(count, torch.int32, "count", (n,))
    ptr = torch.zeros(n + 1, dtype=torch.int64, device=pos.device)
    torch.cumsum(count, 0, out=ptr[1:])
    total = int(ptr[-1].item())
    idx = torch.empty(max(total, 1), dtype=torch.int32, device=pos.device)
    _check(lib.tiga_radius_neighbors(n, _ptr(pos), float(radius), _ptr(ptr), _ptr(idx), _ptr(ws), ws.numel(),
                                     _stream()))
    return count, ptr, idx[:total]


def tiga_mp_dense_fwd(pos: torch.Tensor, q: torch.Tensor, eps: float, y=None, ws=None):
    lib = load()
    n = pos.shape[0]
    _dev(pos, torch.float32, "pos", (n, 3))
    _dev(q, torch.float32, "q", (n,))
    if y is None:
        y = torch.empty(n, 3, dtype=torch.float32, device=pos.device)
    if ws is None:
        ws = _workspace(lib.tiga_mp_dense_workspace(n), pos.device)
    _check(lib.tiga_mp_dense_fwd(n, _ptr(pos), _ptr(q), float(eps), REDUCE_SUM, _ptr(y), _ptr(ws), ws.numel(),
                                 _stream()))
    return y


def _edgenn_args(pos, x, W1, b1, W2, b2):
    n = pos.shape[0]
    _dev(pos, torch.float32, "pos", (n, 3))
    H, D = W1.shape
    F = D - 3
    O = W2.shape[0]
    _dev(W1, torch.float32, "W1", (H, D))
    _dev(b1, torch.float32, "b1", (H,))
    _dev(W2, torch.float32, "W2", (O, H))
    _dev(b2, torch.float32, "b2", (O,))
    if F > 0:
        _dev(x, torch.float32, "x", (n, F))
    return n, F, H, O


def tiga_mp_edgenn_fwd(pos, x, radius, W1, b1, W2, b2, ws=None):
    """y_i = sum over the radius relation of W2 relu(W1 [p_j - p_i; x_j] + b1) + b2; returns y fp32 [n, out]."""
    lib = load()
    n, F, H, O = _edgenn_args(pos, x, W1, b1, W2, b2)
    y = torch.empty(n, O, dtype=torch.float32, device=pos.device)
    if ws is None:
        ws = _workspace(lib.tiga_mp_edgenn_workspace(n, F, H, O), pos.device)
    _check(lib.tiga_mp_edgenn_fwd(n, F, H, O, _ptr(pos), _ptr(x) if F else None, float(radius), _ptr(W1), _ptr(b1),
                                  _ptr(W2), _ptr(b2), _ptr(y), _ptr(ws), ws.numel(), _stream()))
    return y


def tiga_mp_edgenn_bwd(pos, x, radius, W1, b1, W2, b2, dy, want=("dx", "dpos", "dW1", "db1", "dW2", "db2"), ws=None):
    """The VJP of tiga_mp_edgenn_fwd for the cotangent dy [n, out]; returns a dict of the wanted gradients."""
    lib = load()
    n, F, H, O = _edgenn_args(pos, x, W1, b1, W2, b2)
    _dev(dy, torch.float32, "dy", (n, O))
    shapes = dict(dx=(n, F), dpos=(n, 3), dW1=(H, 3 + F), db1=(H,), dW2=(O, H), db2=(O,))
    out = {k: torch.empty(*shapes[k], dtype=torch.float32, device=pos.device) for k in want if shapes[k][-1] > 0}
    if ws is None:
        ws = _workspace(lib.tiga_mp_edgenn_workspace(n, F, H, O), pos.device)
    g = lambda k: _ptr(out.get(k))
    _check(lib.tiga_mp_edgenn_bwd(n, F, H, O, _ptr(pos), _ptr(x) if F else None, float(radius), _ptr(W1), _ptr(b1),
                                  _ptr(W2), _ptr(b2), _ptr(dy), g("dx"), g("dpos"), g("dW1"), g("db1"), g("dW2"),
                                  g("db2"), _ptr(ws), ws.numel(), _stream()))
    return out


def tiga_mp_knn_fwd(pos: torch.Tensor, x: torch.Tensor | None, k: int, want_nbr: bool = False, ws=None):
    """Exact kNN relation (self excluded, key (fp32 d2, index)) with the neighbour sum y_i = sum x_j.

    pos fp32 [n, 3]; x fp32 [n, F] or None.  Returns y fp32 [n, F] (None without x), and the selected
    indices int32 [n, k] in key order when want_nbr."""
    lib = load()
    n = pos.shape[0]
    _dev(pos, torch.float32, "pos", (n, 3))
    F = 0
    if x is not None:
        _dev(x, torch.float32, "x")
        if x.dim() != 2 or x.shape[0] != n:
            raise ValueError(f"x must be [n, F] with n = {n}")
        F = x.shape[1]
    y = torch.empty(n, F, dtype=torch.float32, device=pos.device) if x is not None else None
    nbr = torch.empty(n, k, dtype=torch.int32, device=pos.device) if want_nbr else None
    if ws is None:
        ws = _workspace(lib.tiga_mp_knn_workspace(n), pos.device)
    _check(lib.tiga_mp_knn_fwd(n, F, _ptr(pos), _ptr(x) if F else None, int(k), REDUCE_SUM, _ptr(y) if F else None,
                               _ptr(nbr), _ptr(ws), ws.numel(), _stream()))
    return (y, nbr) if want_nbr else y


def _head_major(t, name, layout, shape=None):
    """The [heads, n, width] storage of t: t itself ("hnd": contiguous [heads, n, width]) or, for "nhd",
    the (n, heads, width) view of a contiguous (heads, n, width) allocation permuted back."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype not in (torch.float16, torch.bfloat16):
        raise TypeError(f"{name} must be float16 or bfloat16, got {t.dtype}")
    if t.dim() != 3:
        raise ValueError(f"{name} must have 3 dimensions")
    if layout == "nhd":
        t = t.permute(1, 0, 2)
    elif layout != "hnd":
        raise ValueError(f"unknown layout {layout!r}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be head-major storage (layout {layout!r})")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has head-major shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def tiga_mp_attention_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, scale: float | None = None,
                          relation: str = "triangular", want_lse: bool = False, layout: str = "hnd"):
    """Online-softmax attention over the triangular (causal, diagonal included) or dense relation.

    q, k, v: float16 or bfloat16, head-major [heads, n, width] (layout "hnd") or the (n, heads, width)
    view of head-major storage (layout "nhd").  scale defaults to width ** -0.5.  Returns y in the
    layout of q (and lse fp32 [heads, n] when want_lse)."""
    lib = load()
    qh = _head_major(q, "q", layout)
    H, n, D = qh.shape
    kh = _head_major(k, "k", layout, (H, n, D))
    vh = _head_major(v, "v", layout, (H, n, D))
    if kh.dtype != qh.dtype or vh.dtype != qh.dtype:
        raise TypeError("q, k and v must share one dtype")
    dt = DT_F16 if qh.dtype == torch.float16 else DT_BF16
    rel = {"triangular": REL_TRIANGULAR, "dense": REL_DENSE}[relation]
    if scale is None:
        scale = D ** -0.5
    yh = torch.empty(H, n, D, dtype=qh.dtype, device=qh.device)
    lse = torch.empty(H, n, dtype=torch.float32, device=qh.device) if want_lse else None
    _check(lib.tiga_mp_attention_fwd(n, H, D, dt, _ptr(qh), _ptr(kh), _ptr(vh), float(scale), rel, _ptr(yh),
                                     _ptr(lse), _stream()))
    y = yh.permute(1, 0, 2) if layout == "nhd" else yh
    return (y, lse) if want_lse else y


# ------------------------------------------------------------ autograd wrappers
#
# The paper's Torch interop (the fused operator as a differentiable function):
# the forward calls the fused entry point, the backward its vector-Jacobian
# product.  The sum saves x and w (dx needs w, dw needs x); max also saves the
# forward's argmax, which routes its gradients.  The relation is a topology
# snapshot: it is not differentiated.


class CsrAggregate(torch.autograd.Function):
    """y = reduce_{e in row i} w[e] * x[col[e]] over a stored CSR relation."""

    @staticmethod
    def forward(ctx, x, w, rel, reducer, rev):
        y, arg = tiga_mp_csr_fwd(rel, x, w, reducer=reducer)
        ctx.rel, ctx.reducer, ctx.rev = rel, reducer, rev
        ctx.save_for_backward(x, w, arg)
        if arg is not None:
            ctx.mark_non_differentiable(arg)
        return y, arg

    @staticmethod
    def backward(ctx, gy, _garg):
        x, w, arg = ctx.saved_tensors
        want_dx = ctx.needs_input_grad[0]
        want_dw = w is not None and ctx.needs_input_grad[1]
        if not (want_dx or want_dw):
            return None, None, None, None, None
        dx, dw = tiga_mp_csr_bwd(ctx.rel, gy.contiguous(), x, w, reducer=ctx.reducer, argmax=arg, rev=ctx.rev,
                                 want_dx=want_dx, want_dw=want_dw)
        return dx, dw, None, None, None


def csr_aggregate(rel: Csr, x: torch.Tensor, w: torch.Tensor | None = None, reducer: int = REDUCE_SUM,
                  rev: CsrT | None = None):
    """Differentiable fused aggregation; returns (y, argmax or None).  With `rev` (the reverse incidence)
    the backward is the deterministic single traversal, without it dx accumulates by atomics."""
    return CsrAggregate.apply(x, w, rel, reducer, rev)


class RadiusAggregate(torch.autograd.Function):
    """y_i = sum_{j != i, |p_j - p_i| < r} exp(-|p_j - p_i|^2 / sigma^2) x_j (membership not differentiated)."""

    @staticmethod
    def forward(ctx, pos, x, radius, sigma):
        y, _ = tiga_mp_radius_fwd(pos, x, radius, sigma, want_count=False)
        ctx.radius, ctx.sigma = radius, sigma
        ctx.save_for_backward(pos, x)
        return y

    @staticmethod
    def backward(ctx, gy):
        pos, x = ctx.saved_tensors
        want_dpos, want_dx = ctx.needs_input_grad[0], ctx.needs_input_grad[1]
        if not (want_dpos or want_dx):
            return None, None, None, None
        dx, dpos = tiga_mp_radius_bwd(pos, x, gy.contiguous(), ctx.radius, ctx.sigma, want_dx=want_dx,
                                      want_dpos=want_dpos)
        return dpos, dx, None, None


def radius_aggregate(pos: torch.Tensor, x: torch.Tensor, radius: float, sigma: float) -> torch.Tensor:
    """Differentiable fused aggregation over the generated radius relation."""
    return RadiusAggregate.apply(pos, x, radius, sigma)


class EdgeMLP(torch.autograd.Function):
    """y = sum over the radius relation of W2 relu(W1 [p_j - p_i; x_j] + b1) + b2 (membership fixed)."""

    @staticmethod
    def forward(ctx, pos, x, W1, b1, W2, b2, radius):
        ctx.radius = radius
        ctx.save_for_backward(pos, x, W1, b1, W2, b2)
        return tiga_mp_edgenn_fwd(pos, x, radius, W1, b1, W2, b2)

    @staticmethod
    def backward(ctx, dy):
        pos, x, W1, b1, W2, b2 = ctx.saved_tensors
        g = tiga_mp_edgenn_bwd(pos, x, ctx.radius, W1, b1, W2, b2, dy.contiguous())
        return g["dpos"], g.get("dx"), g["dW1"], g["db1"], g["dW2"], g["db2"], None


def edge_mlp(pos, x, W1, b1, W2, b2, radius):
    return EdgeMLP.apply(pos, x, W1, b1, W2, b2, radius)
