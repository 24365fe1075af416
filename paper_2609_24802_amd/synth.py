"""Seeded synthetic inputs for fused message passing.

This module only draws inputs: graphs (CSR topology), edge weights, node
features, point clouds, charges and cotangents.  It contains none of the
message-passing arithmetic, so both the HIP path and the CPU oracle can take
their inputs from here without sharing any computation.

Every array is a deterministic function of ``(BASE_SEED, config id, array id,
chunk id)`` through ``numpy.random.SeedSequence(spawn_key=...)``; the result
does not depend on the number of threads used to draw it.

Readings of the workloads (the paper fixes none of these details):

* the base seed is one of the seeds the evaluation protocol names
  (Section 7.5, seeds 20260921-20260923);
* fp32 uniforms are ``a + (b - a) * u`` with ``u = Generator.random(float32)``;
  normals are ``Generator.standard_normal(float32)``;
* a uniform random multigraph is sorted into destination-major CSR with a
  stable sort, so the "edge index" is the CSR position (Section 4.3 uses the
  edge position to index edge fields);
* a power-law in-degree sequence is drawn from ``Generator.zipf(a)``, capped,
  then rescaled to the requested edge count (floor plus largest-remainder),
  re-capping and redistributing until no row exceeds the cap.
"""
from __future__ import annotations

import concurrent.futures as _cf
import hashlib
import math
import os

import numpy as np

BASE_SEED = 20260921
_CHUNK = 1 << 24


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(
        np.random.PCG64(np.random.SeedSequence(BASE_SEED, spawn_key=tuple(int(k) for k in key))))


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _chunked(n: int, key: tuple, fill) -> None:
    """Run ``fill(rng, lo, hi)`` over fixed-size chunks, each with its own stream."""
    nchunk = (n + _CHUNK - 1) // _CHUNK
    if nchunk <= 1:
        if n:
            fill(_rng(*key, 0), 0, n)
        return

    def one(c):
        lo = c * _CHUNK
        fill(_rng(*key, c), lo, min(n, lo + _CHUNK))

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(one, range(nchunk)))


def uniform_f32(n: int, a: float, b: float, key: tuple) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    lo32, span32 = np.float32(a), np.float32(b - a)

    def fill(rng, lo, hi):
        u = rng.random(hi - lo, dtype=np.float32)
        np.multiply(u, span32, out=u)
        np.add(u, lo32, out=out[lo:hi])

    _chunked(n, key, fill)
    return out


def normal_f32(n: int, key: tuple) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)

    def fill(rng, lo, hi):
        rng.standard_normal(hi - lo, dtype=np.float32, out=out[lo:hi])

    _chunked(n, key, fill)
    return out


def randint_i32(n: int, high: int, key: tuple) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)

    def fill(rng, lo, hi):
        out[lo:hi] = rng.integers(0, high, size=hi - lo, dtype=np.int32)

    _chunked(n, key, fill)
    return out


def _largest_remainder(target: np.ndarray, total: int) -> np.ndarray:
    """Integer vector with sum ``total`` closest to the real vector ``target``."""
    base = np.floor(target).astype(np.int64)
    rem = int(total - base.sum())
    if rem > 0:
        frac = target - base
        order = np.argsort(-frac, kind="stable")  # ties -> lower index
        base[order[:rem]] += 1
    return base


def zipf_degrees(n: int, num_edges: int, exponent: float, cap: int, key: tuple) -> np.ndarray:
    """Power-law in-degrees with exactly ``num_edges`` in total, none above ``cap``."""
    if n * cap < num_edges:
        raise ValueError("cap too small for the requested edge count")
    raw = np.minimum(_rng(*key, 0).zipf(exponent, size=n), cap).astype(np.float64)
    deg = _largest_remainder(raw * (num_edges / raw.sum()), num_edges)
    for _ in range(64):
        over = deg > cap
        if not over.any():
            break
        excess = int((deg[over] - cap).sum())
        deg[over] = cap
        free = ~over & (deg < cap)
        share = deg[free].astype(np.float64)
        share = share * (excess / share.sum())
        deg[free] += _largest_remainder(share, excess)
    assert int(deg.sum()) == num_edges and int(deg.max(initial=0)) <= cap
    return deg


def csr_from_degrees(deg: np.ndarray) -> np.ndarray:
    row_ptr = np.zeros(deg.shape[0] + 1, dtype=np.int64)
    np.cumsum(deg, out=row_ptr[1:])
    return row_ptr


def uniform_multigraph_csr(num_dst: int, num_src: int, num_edges: int, key: tuple):
    """(row_ptr int64, col int32, perm) for uniform (src, dst) pairs stably sorted by dst.

    ``perm`` maps CSR position -> generation order, so edge fields drawn in
    generation order can be permuted into CSR order.
    """
    dst = randint_i32(num_edges, num_dst, key + (0,))
    src = randint_i32(num_edges, num_src, key + (1,))
    perm = np.argsort(dst, kind="stable")
    col = src[perm]
    row_ptr = csr_from_degrees(np.bincount(dst, minlength=num_dst).astype(np.int64))
    return row_ptr, col.astype(np.int32), perm


def fingerprint(*arrays: np.ndarray) -> str:
    h = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(memoryview(a.reshape(-1).view(np.uint8)))
    return h.hexdigest()


# ---------------------------------------------------------------------------
# Workloads.  Config ids: 1 small uniform CSR, 2 power-law CSR (1M/16M/F64),
# 3 radius point cloud (1M, F32), 4 dense particles (65,536), 5 power-law
# CSR (50M/1e9/F16).  ``scale`` shrinks a workload for quick runs while keeping
# its shape and distributions.
# ---------------------------------------------------------------------------

def csr_uniform_small(num_nodes=1024, num_edges=8192, feat=16, cfg=1):
    row_ptr, col, perm = uniform_multigraph_csr(num_nodes, num_nodes, num_edges, (cfg, 0))
    w = uniform_f32(num_edges, 0.0, 1.0, (cfg, 1))[perm]
    x = uniform_f32(num_nodes * feat, -1.0, 1.0, (cfg, 2)).reshape(num_nodes, feat)
    dy = normal_f32(num_nodes * feat, (cfg, 3)).reshape(num_nodes, feat)
    return dict(row_ptr=row_ptr, col=col, w=w, x=x, dy=dy, num_dst=num_nodes, num_src=num_nodes)


def csr_powerlaw(num_nodes, num_edges, feat, cap, exponent=2.1, cfg=2, with_dy=True):
    deg = zipf_degrees(num_nodes, num_edges, exponent, cap, (cfg, 0))
    row_ptr = csr_from_degrees(deg)
    del deg
    col = randint_i32(num_edges, num_nodes, (cfg, 1))
    w = uniform_f32(num_edges, 0.0, 1.0, (cfg, 2))
    x = normal_f32(num_nodes * feat, (cfg, 3)).reshape(num_nodes, feat)
    out = dict(row_ptr=row_ptr, col=col, w=w, x=x, num_dst=num_nodes, num_src=num_nodes)
    if with_dy:
        out["dy"] = normal_f32(num_nodes * feat, (cfg, 4)).reshape(num_nodes, feat)
    return out


def config2(scale: float = 1.0):
    n = max(64, int(1_000_000 * scale))
    return csr_powerlaw(n, 16 * n, 64, cap=max(8, int(100_000 * scale)), cfg=2)


def config5(scale: float = 1.0, with_dy: bool = False):
    n = max(64, int(50_000_000 * scale))
    return csr_powerlaw(n, 20 * n, 16, cap=max(8, int(1_000_000 * scale)), cfg=5, with_dy=with_dy)


def radius_for_mean_degree(n: int, mean_degree: float = 32.0) -> np.float32:
    """r with (4/3) pi r^3 n = mean_degree, evaluated in fp64 and rounded to fp32."""
    return np.float32((mean_degree * 3.0 / (4.0 * math.pi * n)) ** (1.0 / 3.0))


def config3(n: int = 1_000_000, feat: int = 32, cfg=3):
    pos = uniform_f32(n * 3, 0.0, 1.0, (cfg, 0)).reshape(n, 3)
    x = normal_f32(n * feat, (cfg, 1)).reshape(n, feat)
    dy = normal_f32(n * feat, (cfg, 2)).reshape(n, feat)
    r = radius_for_mean_degree(n)
    return dict(pos=pos, x=x, dy=dy, radius=r, sigma=np.float32(r / np.float32(2)))


def config4(n: int = 65_536, cfg=4):
    pos = normal_f32(n * 3, (cfg, 0)).reshape(n, 3)
    q = uniform_f32(n, 0.5, 1.5, (cfg, 1))
    return dict(pos=pos, q=q, eps=np.float32(1e-2))


def csr_fixed_degree(num_nodes: int, degree: int, feat: int, cfg: int = 9):
    """Every destination has `degree` edges from uniform sources (the stored-CSR workload of the
    paper's latency experiments): x ~ N(0, 1) [num_nodes, feat], w ~ U(0, 1)."""
    E = num_nodes * degree
    row_ptr = csr_from_degrees(np.full(num_nodes, degree, dtype=np.int64))
    col = randint_i32(E, num_nodes, (cfg, num_nodes, 0))
    w = uniform_f32(E, 0.0, 1.0, (cfg, num_nodes, 1))
    x = normal_f32(num_nodes * feat, (cfg, num_nodes, 2)).reshape(num_nodes, feat)
    return dict(row_ptr=row_ptr, col=col, w=w, x=x, num_dst=num_nodes, num_src=num_nodes)


def binary_grid_points(n: int, bits: int, key: tuple, span: int | None = None) -> np.ndarray:
    """Points whose coordinates are multiples of 2**-bits in [0, span * 2**-bits)."""
    span = span if span is not None else (1 << bits)
    k = _rng(*key, 0).integers(0, span, size=(n, 3))
    return (k.astype(np.float64) * 2.0 ** -bits).astype(np.float32)


def f32_to_half_bits(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp32 values to binary16 ("f16") or bfloat16 ("bf16") with round-to-nearest-even and
    return the 16-bit patterns (uint16).  Input preparation only: finite inputs."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f16":
        return a.astype(np.float16).view(np.uint16)
    if dtype == "bf16":
        u = a.view(np.uint32).astype(np.uint64)
        u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
        return u.astype(np.uint16)
    raise ValueError(dtype)


def attention_inputs(n: int, heads: int, width: int, dtype: str = "f16", cfg: int = 6, sigma: float = 1.0):
    """Head-major [heads, n, width] query, key and value bit patterns, each drawn as sigma * N(0, 1)
    in fp32 and rounded to `dtype`; scale = width ** -0.5 (the causal-attention example of the
    appendix draws torch.randn in head-major storage and uses this scale)."""
    out = {}
    for a, name in enumerate(("q", "k", "v")):
        x = normal_f32(heads * n * width, (cfg, a, n, heads, width))
        if sigma != 1.0:
            x *= np.float32(sigma)
        out[name] = f32_to_half_bits(x, dtype).reshape(heads, n, width)
    out["scale"] = np.float32(width ** -0.5)
    out["dtype"] = dtype
    return out


def knn_inputs(n: int, feat: int = 1, cfg: int = 7):
    """Points uniform in [0, 1)^3 and N(0, 1) features [n, feat]: the exact-kNN workload of the
    evaluation (a scalar neighbour sum, k = 16, 1,024 to 131,072 points)."""
    pos = uniform_f32(n * 3, 0.0, 1.0, (cfg, 0, n)).reshape(n, 3)
    x = normal_f32(n * feat, (cfg, 1, n, feat)).reshape(n, feat)
    return dict(pos=pos, x=x, k=16)


def surface_points(n: int, key: tuple, axes=(0.5, 0.45, 0.40)) -> np.ndarray:
    """Points on an ellipsoid surface (directions uniform on the sphere, scaled by the semi-axes),
    centred and divided by the largest bounding-box extent: a closed-surface cloud standing in for
    a scanned surface mesh's vertices."""
    d = normal_f32(n * 3, key).reshape(n, 3).astype(np.float64)
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    p = d * np.asarray(axes, np.float64)
    p -= 0.5 * (p.min(0) + p.max(0))
    p /= (p.max(0) - p.min(0)).max()
    return p.astype(np.float32)


def mlp_params(fan_in: int, hidden: int, out: int, key: tuple):
    """Weights of Linear(fan_in, hidden) -> ReLU -> Linear(hidden, out), each entry uniform in
    +-1/sqrt(fan in) of its layer (the usual untrained initialization)."""
    b1 = 1.0 / math.sqrt(fan_in)
    b2 = 1.0 / math.sqrt(hidden)
    return dict(W1=uniform_f32(hidden * fan_in, -b1, b1, key + (0,)).reshape(hidden, fan_in),
                b1=uniform_f32(hidden, -b1, b1, key + (1,)),
                W2=uniform_f32(out * hidden, -b2, b2, key + (2,)).reshape(out, hidden),
                b2=uniform_f32(out, -b2, b2, key + (3,)))


def edgenn_inputs(n: int = 35947, feat: int = 8, hidden: int = 32, out: int = 3, radius: float = 0.015, cfg: int = 8):
    """The differentiated edge-MLP workload: surface points (35,947 of them, the size of the scanned
    surface the evaluation uses), radius 0.015, N(0, 1) features of width 8 or 32, an untrained
    MLP (3 + feat) -> hidden -> out, and an N(0, 1) output cotangent."""
    pos = surface_points(n, (cfg, 0, n))
    x = normal_f32(n * feat, (cfg, 1, n, feat)).reshape(n, feat)
    prm = mlp_params(3 + feat, hidden, out, (cfg, 2, feat, hidden, out))
    dy = normal_f32(n * out, (cfg, 3, n, out)).reshape(n, out)
    return dict(pos=pos, x=x, radius=np.float32(radius), dy=dy, **prm)
