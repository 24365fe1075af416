// Generated radius relation (Section 4.9 of the paper): a uniform cell
// directory restricts candidates, an exact fp32 distance predicate accepts,
// and accepted messages are folded into registers without storing edges.
//
// Build (every call, stateless):
//   bounding box -> cell size h >= r (1 + 2^-10), at most n + 64 cells ->
//   cell id per point (fp64 coordinates) -> counts -> exclusive scan ->
//   scatter (counting sort) -> per-cell sort by point id (deterministic order)
//   -> cell-ordered records (p, id) and feature rows.
// Consume: one thread per destination point in cell order; the 27 neighbour
// cells are 9 contiguous runs of the cell-ordered arrays (x-adjacent cells are
// adjacent in memory).
#include "csr_bwd.hpp"
#include "radius.hpp"

namespace tiga {
namespace radius {

using csr::launch_excl_scan;
using csr::scan_ws_bytes;

namespace {

constexpr int kBlock = 256;

struct Params {
    double lo[3];
    double inv_h;
    int dim[3];
    int ncell;
};

__global__ __launch_bounds__(kBlock) void bbox_partial_kernel(const float *__restrict__ pos, int64_t n,
                                                              float *__restrict__ part) {
    float mn[3] = {__builtin_inff(), __builtin_inff(), __builtin_inff()};
    float mx[3] = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            const float v = pos[i * 3 + a];
            mn[a] = fminf(mn[a], v);
            mx[a] = fmaxf(mx[a], v);
        }
    }
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1)
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            mn[a] = fminf(mn[a], shfl_xor_f(mn[a], m));
            mx[a] = fmaxf(mx[a], shfl_xor_f(mx[a], m));
        }
    __shared__ float sh[kBlock / kWave][6];
    const int wave = threadIdx.x / kWave;
    if (lane_id() == 0)
        for (int a = 0; a < 3; ++a) {
            sh[wave][a] = mn[a];
            sh[wave][3 + a] = mx[a];
        }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kBlock / kWave; ++w)
            for (int a = 0; a < 3; ++a) {
                sh[0][a] = fminf(sh[0][a], sh[w][a]);
                sh[0][3 + a] = fmaxf(sh[0][3 + a], sh[w][3 + a]);
            }
        for (int k = 0; k < 6; ++k) part[blockIdx.x * 6 + k] = sh[0][k];
    }
}

// One thread: final box, cell size and grid dimensions.
__global__ void grid_params_kernel(const float *__restrict__ part, int nblocks, int64_t n, float radius,
                                   int64_t max_cells, Params *__restrict__ prm) {
    double lo[3], hi[3];
    for (int a = 0; a < 3; ++a) {
        lo[a] = __builtin_inf();
        hi[a] = -__builtin_inf();
    }
    for (int b = 0; b < nblocks; ++b)
        for (int a = 0; a < 3; ++a) {
            lo[a] = fmin(lo[a], static_cast<double>(part[b * 6 + a]));
            hi[a] = fmax(hi[a], static_cast<double>(part[b * 6 + 3 + a]));
        }
    double ext[3], vol = 1.0;
    for (int a = 0; a < 3; ++a) {
        ext[a] = hi[a] - lo[a];
        if (!(ext[a] >= 0.0)) ext[a] = 0.0;
        vol *= ext[a];
    }
    // cells no smaller than the radius (with a relative margin that covers the
    // fp32 rounding of the predicate), and not much smaller than the mean
    // point spacing
    double h = static_cast<double>(radius) * (1.0 + 1.0 / 1024.0);
    const double spacing = cbrt(vol / static_cast<double>(n > 0 ? n : 1));
    if (spacing > h) h = spacing;
    int64_t d[3];
    for (int it = 0; it < 200; ++it) {
        int64_t cells = 1;
        for (int a = 0; a < 3; ++a) {
            const double t = floor(ext[a] / h) + 1.0;
            d[a] = t > 2e9 ? static_cast<int64_t>(2e9) : static_cast<int64_t>(t);
            cells = (cells > (int64_t{1} << 40)) ? cells : cells * d[a];
        }
        if (cells <= max_cells) break;
        h *= 1.25;
    }
    for (int a = 0; a < 3; ++a) {
        prm->lo[a] = lo[a];
        prm->dim[a] = static_cast<int>(d[a]);
    }
    prm->inv_h = 1.0 / h;
    prm->ncell = static_cast<int>(d[0] * d[1] * d[2]);
}

__device__ __forceinline__ int cell_axis(const Params &p, int a, float v) {
    double t = floor((static_cast<double>(v) - p.lo[a]) * p.inv_h);
    int c = static_cast<int>(t);
    if (t < 0.0) c = 0;
    if (c >= p.dim[a]) c = p.dim[a] - 1;
    return c;
}

__global__ __launch_bounds__(kBlock) void cell_count_kernel(const float *__restrict__ pos, int64_t n,
                                                            const Params *__restrict__ prm,
                                                            int32_t *__restrict__ cell,
                                                            unsigned long long *__restrict__ count) {
    const Params p = *prm;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int cx = cell_axis(p, 0, pos[i * 3 + 0]);
        const int cy = cell_axis(p, 1, pos[i * 3 + 1]);
        const int cz = cell_axis(p, 2, pos[i * 3 + 2]);
        const int c = (cz * p.dim[1] + cy) * p.dim[0] + cx;
        cell[i] = c;
        atomicAdd(&count[c], 1ull);
    }
}

__global__ __launch_bounds__(kBlock) void cell_scatter_kernel(const int32_t *__restrict__ cell, int64_t n,
                                                              const int64_t *__restrict__ start,
                                                              unsigned int *__restrict__ cursor,
                                                              int32_t *__restrict__ perm) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int c = cell[i];
        perm[start[c] + atomicAdd(&cursor[c], 1u)] = static_cast<int32_t>(i);
    }
}

// Sort the point ids of each cell ascending so that the candidate order (and
// hence every summation order) depends only on the input.  A wavefront per
// cell computes each element's rank; cells beyond kSortMax points keep the
// order of the scatter (still correct, not bit-reproducible).
constexpr int kSortMax = 4096;

__global__ __launch_bounds__(kBlock) void cell_sort_kernel(const int64_t *__restrict__ start,
                                                           const Params *__restrict__ prm,
                                                           const int32_t *__restrict__ perm_in,
                                                           int32_t *__restrict__ perm_out) {
    const int ncell = prm->ncell;
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * (kBlock / kWave) + threadIdx.x / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
    for (int64_t c = wave; c < ncell; c += nwaves) {
        const int64_t b = start[c], e = start[c + 1], d = e - b;
        if (d > kSortMax) {
            for (int64_t k = b + lane_id(); k < e; k += kWave) perm_out[k] = perm_in[k];
            continue;
        }
        for (int64_t k = b + lane_id(); k < e; k += kWave) {
            const int32_t v = perm_in[k];
            int64_t rank = 0;
            for (int64_t m = b; m < e; ++m) rank += perm_in[m] < v;
            perm_out[b + rank] = v;
        }
    }
}

// Cell-ordered records and feature rows.
__global__ __launch_bounds__(kBlock) void gather_sorted_kernel(const int32_t *__restrict__ perm, int64_t n,
                                                               const float *__restrict__ pos,
                                                               const float *__restrict__ a, const float *__restrict__ b,
                                                               int32_t feat, float4 *__restrict__ rec,
                                                               float *__restrict__ as, float *__restrict__ bs) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; s < n; s += stride) {
        const int32_t i = perm[s];
        rec[s] = make_float4(pos[i * 3 + 0], pos[i * 3 + 1], pos[i * 3 + 2], __int_as_float(i));
    }
    // feature rows: one element per thread, coalesced on the destination
    const int64_t total = n * feat;
    for (int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; k < total; k += stride) {
        const int64_t s = k / feat;
        const int64_t f = k - s * feat;
        const int64_t i = perm[s];
        if (a) as[k] = a[i * feat + f];
        if (b) bs[k] = b[i * feat + f];
    }
}

// Exact membership test: direct fp32 differences, products and sums, each
// rounded once (no contraction), strict comparison with fp32(r*r).
__device__ __forceinline__ bool accept(float4 pi, float4 pj, float r2, float &d2) {
#pragma clang fp contract(off)
    const float dx = pj.x - pi.x;
    const float dy = pj.y - pi.y;
    const float dz = pj.z - pi.z;
    const float sx = dx * dx;
    const float sy = dy * dy;
    const float sz = dz * dz;
    d2 = (sx + sy) + sz;
    return d2 < r2;
}

// Visit the candidate runs of the point with record `pi`.
template <class F>
__device__ __forceinline__ void for_candidates(const Params &p, const int64_t *__restrict__ start, float4 pi,
                                               F &&body) {
    const int cx = cell_axis(p, 0, pi.x);
    const int cy = cell_axis(p, 1, pi.y);
    const int cz = cell_axis(p, 2, pi.z);
    const int x0 = cx > 0 ? cx - 1 : 0;
    const int x1 = cx + 1 < p.dim[0] ? cx + 1 : p.dim[0] - 1;
    for (int z = cz - 1; z <= cz + 1; ++z) {
        if (z < 0 || z >= p.dim[2]) continue;
        for (int y = cy - 1; y <= cy + 1; ++y) {
            if (y < 0 || y >= p.dim[1]) continue;
            const int rowc = (z * p.dim[1] + y) * p.dim[0];
            const int64_t b = start[rowc + x0];
            const int64_t e = start[rowc + x1 + 1];
            for (int64_t t = b; t < e; ++t) body(t);
        }
    }
}

// FB float4 units of features per pass (a feature block), scalar tail handled
// by the K = 1 instantiation.
template <int K, int NU>
__global__ __launch_bounds__(kBlock) void radius_fwd_kernel(const Params *__restrict__ prm,
                                                            const int64_t *__restrict__ start,
                                                            const float4 *__restrict__ rec,
                                                            const float *__restrict__ xs, int64_t n, int64_t fu,
                                                            float r2, float neg_inv_s2, float *__restrict__ y,
                                                            int32_t *__restrict__ count) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    for (int64_t fb = 0; fb < fu; fb += NU) {
        float acc[NU][K];
#pragma unroll
        for (int u = 0; u < NU; ++u)
#pragma unroll
            for (int k = 0; k < K; ++k) acc[u][k] = 0.0f;
        int cnt = 0;
        for_candidates(p, start, pi, [&](int64_t t) {
            const float4 pj = rec[t];
            float d2;
            if (accept(pi, pj, r2, d2) && __float_as_int(pj.w) != i) {
                ++cnt;
                const float kw = __expf(d2 * neg_inv_s2);
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    if (fb + u < fu) {
                        csr::Vec<K> xv = csr::load_unit<K>(xs, t * fu + fb + u);
#pragma unroll
                        for (int k = 0; k < K; ++k) acc[u][k] = fmaf(kw, xv.v[k], acc[u][k]);
                    }
                }
            }
        });
#pragma unroll
        for (int u = 0; u < NU; ++u)
            if (fb + u < fu) csr::store_unit<K>(y, static_cast<int64_t>(i) * fu + fb + u, acc[u]);
        if (fb == 0 && count) count[i] = cnt;
    }
}

// Backward: dx_i = sum k_ij dy_j and dp_i = sum (2 k_ij / sigma^2)(p_j - p_i)
// (<dy_i, x_j> + <dy_j, x_i>), one thread per destination point.
template <int K, int NU, bool DX, bool DP>
__global__ __launch_bounds__(kBlock) void radius_bwd_kernel(const Params *__restrict__ prm,
                                                            const int64_t *__restrict__ start,
                                                            const float4 *__restrict__ rec,
                                                            const float *__restrict__ xs,
                                                            const float *__restrict__ ys, int64_t n, int64_t fu,
                                                            float r2, float neg_inv_s2, float two_inv_s2,
                                                            float *__restrict__ dx, float *__restrict__ dp) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    float gp[3] = {0.0f, 0.0f, 0.0f};
    for (int64_t fb = 0; fb < fu; fb += NU) {
        float gi[NU][K], xi[NU][K], acc[NU][K];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            csr::Vec<K> a, b;
            if (fb + u < fu) {
                a = csr::load_unit<K>(ys, s * fu + fb + u);
                if (DP) {
                    b = csr::load_unit<K>(xs, s * fu + fb + u);
                } else {
#pragma unroll
                    for (int k = 0; k < K; ++k) b.v[k] = 0.0f;
                }
            } else {
#pragma unroll
                for (int k = 0; k < K; ++k) a.v[k] = b.v[k] = 0.0f;
            }
#pragma unroll
            for (int k = 0; k < K; ++k) {
                gi[u][k] = a.v[k];
                xi[u][k] = b.v[k];
                acc[u][k] = 0.0f;
            }
        }
        float blk[3] = {0.0f, 0.0f, 0.0f};
        for_candidates(p, start, pi, [&](int64_t t) {
            const float4 pj = rec[t];
            float d2;
            if (accept(pi, pj, r2, d2) && __float_as_int(pj.w) != i) {
                const float kw = __expf(d2 * neg_inv_s2);
                float dot = 0.0f;
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    if (fb + u < fu) {
                        csr::Vec<K> gj = csr::load_unit<K>(ys, t * fu + fb + u);
                        csr::Vec<K> xj;
                        if (DP) xj = csr::load_unit<K>(xs, t * fu + fb + u);
#pragma unroll
                        for (int k = 0; k < K; ++k) {
                            if (DX) acc[u][k] = fmaf(kw, gj.v[k], acc[u][k]);
                            if (DP) dot = fmaf(gi[u][k], xj.v[k], fmaf(gj.v[k], xi[u][k], dot));
                        }
                    }
                }
                if (DP) {
                    const float c = two_inv_s2 * kw * dot;
                    blk[0] = fmaf(c, pj.x - pi.x, blk[0]);
                    blk[1] = fmaf(c, pj.y - pi.y, blk[1]);
                    blk[2] = fmaf(c, pj.z - pi.z, blk[2]);
                }
            }
        });
        if (DX) {
#pragma unroll
            for (int u = 0; u < NU; ++u)
                if (fb + u < fu) csr::store_unit<K>(dx, static_cast<int64_t>(i) * fu + fb + u, acc[u]);
        }
        gp[0] += blk[0];
        gp[1] += blk[1];
        gp[2] += blk[2];
    }
    if (DP) {
        dp[static_cast<int64_t>(i) * 3 + 0] = gp[0];
        dp[static_cast<int64_t>(i) * 3 + 1] = gp[1];
        dp[static_cast<int64_t>(i) * 3 + 2] = gp[2];
    }
}

__global__ __launch_bounds__(kBlock) void neighbor_count_kernel(const Params *__restrict__ prm,
                                                                const int64_t *__restrict__ start,
                                                                const float4 *__restrict__ rec, int64_t n, float r2,
                                                                int64_t *__restrict__ cnt64,
                                                                int32_t *__restrict__ count) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    int c = 0;
    for_candidates(p, start, pi, [&](int64_t t) {
        const float4 pj = rec[t];
        float d2;
        if (accept(pi, pj, r2, d2) && __float_as_int(pj.w) != i) ++c;
    });
    cnt64[i] = c;
    if (count) count[i] = c;
}

__global__ __launch_bounds__(kBlock) void neighbor_fill_kernel(const Params *__restrict__ prm,
                                                               const int64_t *__restrict__ start,
                                                               const float4 *__restrict__ rec, int64_t n, float r2,
                                                               const int64_t *__restrict__ ptr,
                                                               int32_t *__restrict__ idx) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    const int64_t b = ptr[i];
    int64_t w = b;
    for_candidates(p, start, pi, [&](int64_t t) {
        const float4 pj = rec[t];
        float d2;
        const int32_t j = __float_as_int(pj.w);
        if (accept(pi, pj, r2, d2) && j != i) idx[w++] = j;
    });
    // insertion sort of this point's list (ascending ids)
    for (int64_t a = b + 1; a < w; ++a) {
        const int32_t v = idx[a];
        int64_t k = a - 1;
        while (k >= b && idx[k] > v) {
            idx[k + 1] = idx[k];
            --k;
        }
        idx[k + 1] = v;
    }
}

struct Ws {
    Params *prm;
    float *bbox;
    int32_t *cell;
    unsigned long long *count;  // ncell_max + 1, scanned in place into `start`
    unsigned int *cursor;
    int32_t *perm_a, *perm_b;
    float4 *rec;
    float *as, *bs;
    void *scan;
    int64_t max_cells;
    int bbox_blocks;
};

Ws carve(Carve &c, int64_t n, int64_t feat) {
    Ws w;
    w.max_cells = n + 64;
    w.bbox_blocks = 1024;
    w.prm = c.take<Params>(1);
    w.bbox = c.take<float>(6 * w.bbox_blocks);
    w.cell = c.take<int32_t>(n);
    w.count = c.take<unsigned long long>(w.max_cells + 1);
    w.cursor = c.take<unsigned int>(w.max_cells);
    w.perm_a = c.take<int32_t>(n);
    w.perm_b = c.take<int32_t>(n);
    w.rec = c.take<float4>(n);
    w.as = c.take<float>(n * feat);
    w.bs = c.take<float>(n * feat);
    w.scan = c.take<char>(scan_ws_bytes(w.max_cells + 1));
    return w;
}

int blocks_for(int64_t n) {
    int64_t b = ceil_div(n > 0 ? n : 1, kBlock);
    const int64_t cap = static_cast<int64_t>(device_cus()) * 32;
    return static_cast<int>(b < cap ? b : cap);
}

// Build the cell directory and the cell-ordered copies of `a` and `b`.
int build(int64_t n, const float *pos, float radius, const float *a, const float *b, int32_t feat, Ws &w,
          hipStream_t stream) {
    int nb = w.bbox_blocks;
    const int64_t need = ceil_div(n, kBlock);
    if (need < nb) nb = static_cast<int>(need);
    hipLaunchKernelGGL(bbox_partial_kernel, dim3(nb), dim3(kBlock), 0, stream, pos, n, w.bbox);
    if (int rc = check_launch("radius bbox")) return rc;
    hipLaunchKernelGGL(grid_params_kernel, dim3(1), dim3(1), 0, stream, w.bbox, nb, n, radius, w.max_cells, w.prm);
    if (int rc = check_launch("radius grid")) return rc;
    if (int rc = fill_u32(w.count, 0u, 2 * (w.max_cells + 1), stream)) return rc;
    if (int rc = fill_u32(w.cursor, 0u, w.max_cells, stream)) return rc;
    hipLaunchKernelGGL(cell_count_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, pos, n, w.prm, w.cell,
                       w.count);
    if (int rc = check_launch("radius cell count")) return rc;
    int64_t *start = reinterpret_cast<int64_t *>(w.count);
    if (int rc = launch_excl_scan(start, start, w.max_cells + 1, w.scan, stream)) return rc;
    hipLaunchKernelGGL(cell_scatter_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, w.cell, n, start,
                       w.cursor, w.perm_a);
    if (int rc = check_launch("radius scatter")) return rc;
    hipLaunchKernelGGL(cell_sort_kernel, dim3(blocks_for(w.max_cells * kWave)), dim3(kBlock), 0, stream, start, w.prm,
                       w.perm_a, w.perm_b);
    if (int rc = check_launch("radius cell sort")) return rc;
    hipLaunchKernelGGL(gather_sorted_kernel, dim3(blocks_for(n * (feat > 0 ? feat : 1))), dim3(kBlock), 0, stream,
                       w.perm_b, n, pos, a, b, feat, w.rec, w.as, w.bs);
    return check_launch("radius gather");
}

template <int K>
int fwd_units(int64_t fu, const Ws &w, const int64_t *start, int64_t n, float r2, float nis, float *y,
              int32_t *count, hipStream_t stream) {
    const dim3 grid(static_cast<unsigned>(ceil_div(n, kBlock)));
#define TIGA_RF(NU)                                                                                            \
    hipLaunchKernelGGL((radius_fwd_kernel<K, NU>), grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, w.as, n, \
                       fu, r2, nis, y, count)
    prof_before(stream);
    if (fu <= 1) TIGA_RF(1);
    else if (fu <= 2) TIGA_RF(2);
    else if (fu <= 4) TIGA_RF(4);
    else if (fu <= 8) TIGA_RF(8);
    else TIGA_RF(16);
#undef TIGA_RF
    prof_after(stream);
    return check_launch("radius forward");
}

template <int K, bool DX, bool DP>
int bwd_units(int64_t fu, const Ws &w, const int64_t *start, int64_t n, float r2, float nis, float tis, float *dx,
              float *dp, hipStream_t stream) {
    const dim3 grid(static_cast<unsigned>(ceil_div(n, kBlock)));
#define TIGA_RB(NU)                                                                                          \
    hipLaunchKernelGGL((radius_bwd_kernel<K, NU, DX, DP>), grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, \
                       w.bs, w.as, n, fu, r2, nis, tis, dx, dp)
    prof_before(stream);
    if (fu <= 1) TIGA_RB(1);
    else if (fu <= 2) TIGA_RB(2);
    else if (fu <= 4) TIGA_RB(4);
    else TIGA_RB(8);
#undef TIGA_RB
    prof_after(stream);
    return check_launch("radius backward");
}

}  // namespace

size_t workspace_bytes(int64_t n, int64_t feat) {
    Carve c(nullptr);
    carve(c, n, feat);
    return c.bytes();
}

int forward(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma, float *y,
            int32_t *count, void *ws, hipStream_t stream) {
    Carve c(ws);
    Ws w = carve(c, n, feat);
    if (int rc = build(n, pos, radius, x, nullptr, feat, w, stream)) return rc;
    const int64_t *start = reinterpret_cast<const int64_t *>(w.count);
    const float r2 = radius * radius;
    const float nis = -1.0f / (sigma * sigma);
    const bool vec = feat % 4 == 0 && aligned16(y);
    if (vec) return fwd_units<4>(feat / 4, w, start, n, r2, nis, y, count, stream);
    return fwd_units<1>(feat, w, start, n, r2, nis, y, count, stream);
}

int backward(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma, const float *dy,
             float *dx, float *dpos, void *ws, hipStream_t stream) {
    Carve c(ws);
    Ws w = carve(c, n, feat);
    // as = cell-ordered dy, bs = cell-ordered x (only needed for dpos)
    if (int rc = build(n, pos, radius, dy, dpos ? x : nullptr, feat, w, stream)) return rc;
    const int64_t *start = reinterpret_cast<const int64_t *>(w.count);
    const float r2 = radius * radius;
    const float nis = -1.0f / (sigma * sigma);
    const float tis = 2.0f / (sigma * sigma);
    const bool vec = feat % 4 == 0 && (!dx || aligned16(dx));
    const int64_t fu = vec ? feat / 4 : feat;
#define TIGA_B(KK)                                                                          \
    if (dx && dpos) return bwd_units<KK, true, true>(fu, w, start, n, r2, nis, tis, dx, dpos, stream); \
    if (dx) return bwd_units<KK, true, false>(fu, w, start, n, r2, nis, tis, dx, dpos, stream);        \
    return bwd_units<KK, false, true>(fu, w, start, n, r2, nis, tis, dx, dpos, stream)
    if (vec) {
        TIGA_B(4);
    } else {
        TIGA_B(1);
    }
#undef TIGA_B
}

int neighbors(int64_t n, const float *pos, float radius, int32_t *count, int64_t *nbr_ptr, int32_t *nbr_idx,
              void *ws, hipStream_t stream) {
    Carve c(ws);
    Ws w = carve(c, n, 0);
    if (int rc = build(n, pos, radius, nullptr, nullptr, 0, w, stream)) return rc;
    const int64_t *start = reinterpret_cast<const int64_t *>(w.count);
    const float r2 = radius * radius;
    const dim3 grid(static_cast<unsigned>(ceil_div(n, kBlock)));
    if (!nbr_idx) {
        // counts into nbr_ptr[0..n), then the exclusive scan in place
        hipLaunchKernelGGL(neighbor_count_kernel, grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, n, r2, nbr_ptr,
                           count);
        if (int rc = check_launch("radius neighbour count")) return rc;
        if (int rc = fill_u32(nbr_ptr + n, 0u, 2, stream)) return rc;
        if (int rc = launch_excl_scan(nbr_ptr, nbr_ptr, n + 1, w.scan, stream)) return rc;
    } else {
        hipLaunchKernelGGL(neighbor_fill_kernel, grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, n, r2, nbr_ptr,
                           nbr_idx);
        if (int rc = check_launch("radius neighbour fill")) return rc;
    }
    return check_hip(hipStreamSynchronize(stream), "radius neighbours: synchronize");
}

}  // namespace radius
}  // namespace tiga
